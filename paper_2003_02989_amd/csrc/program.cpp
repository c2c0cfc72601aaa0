// program.cpp -- parsing, validation, structure dedupe and pass planning.
//
// Planning follows the idea behind the paper's gate fusion (Sec. "Gate Fusion
// with qsim"): every application of a gate costs a sweep over all 2^n
// amplitudes, so as many gates as possible are applied per sweep.  Here a
// sweep is a "tile pass": each workgroup stages a tile of 2^t amplitudes in
// LDS (t index bits: the lowest `low` bits, for coalesced HBM runs, plus
// chosen high bits), applies every gate of the pass whose non-diagonal qubits
// lie in the tile -- diagonal gates and control qubits may sit outside, their
// bit is then constant over the tile -- and writes the tile back.  Inside a
// pass, neighbouring gates on the same qubit set are pre-multiplied into one
// matrix on the device.
#include "program.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <set>

#include "../../include/tq.h"

namespace tq {

namespace {

struct Reader {
    const uint8_t *p, *end;
    bool bad = false;
    template <class T> T get()
    {
        T v{};
        if (end - p < (long)sizeof(T)) {
            bad = true;
            return v;
        }
        std::memcpy(&v, p, sizeof(T));
        p += sizeof(T);
        return v;
    }
};

[[noreturn]] void fail(int status, const std::string &m) { throw Error{status, m}; }

bool op_shape(int op, int &nq, int &np)
{
    switch (op) {
    case OP_H: case OP_X: case OP_Y: case OP_Z: case OP_SQRTX: case OP_SQRTY: case OP_SQRTW: case OP_MATRIX1:
        nq = 1; np = 0; return true;
    case OP_RX: case OP_RY: case OP_RZ: case OP_XPOW: case OP_YPOW: case OP_ZPOW:
        nq = 1; np = 1; return true;
    case OP_CZ: case OP_CNOT: case OP_MATRIX2: case OP_SWAP:
        nq = 2; np = 0; return true;
    case OP_CZPOW: case OP_CNOTPOW: case OP_XXPOW: case OP_YYPOW: case OP_ZZPOW: case OP_RZZ:
        nq = 2; np = 1; return true;
    case OP_FSIM:
        nq = 2; np = 2; return true;
    case OP_PCHAN:
        nq = 1; np = 3; return true;
    default:
        return false;
    }
}

// Gate classes as the tile passes see them.
enum Cls { C_1D, C_1M, C_CTRL, C_2D, C_2M, C_2P, C_2F };

int classify(int op)
{
    switch (op) {
    case OP_Z: case OP_RZ: case OP_ZPOW:
        return C_1D;
    case OP_CNOT: case OP_CNOTPOW:
        return C_CTRL;
    case OP_CZ: case OP_CZPOW: case OP_ZZPOW: case OP_RZZ:
        return C_2D;
    case OP_XXPOW: case OP_YYPOW:
        return C_2P;
    case OP_FSIM: case OP_SWAP:
        return C_2F;
    case OP_MATRIX2:
        return C_2M;
    default:
        return C_1M;
    }
}

// Qubits whose bit must be local to the tile (the non-diagonal ones).
int targets(const Group &g, int gi, int *out)
{
    int cls = classify(g.gates[gi].op);
    switch (cls) {
    case C_1D: case C_2D: return 0;
    case C_1M: out[0] = g.gate_q0[gi]; return 1;
    case C_CTRL: out[0] = g.gate_q1[gi]; return 1;
    default: out[0] = g.gate_q0[gi]; out[1] = g.gate_q1[gi]; return 2;
    }
}

int qubits_of(const Group &g, int gi, int *out)
{
    out[0] = g.gate_q0[gi];
    if (g.gates[gi].nq == 2) {
        out[1] = g.gate_q1[gi];
        return 2;
    }
    return 1;
}

// Tile-bit swaps the pass scheduler tries per pass (each one places more gates).
constexpr int kTileSearchSteps = 64;

struct Sched {
    std::vector<int> bits;   // tile bit positions
    std::vector<int> items;  // gate indices in application order
};

// Greedy pass scheduling.  A gate joins the current pass when none of its
// qubits is blocked by an earlier deferred gate and its target bits fit in
// the tile (choosing new tile bits while there is room); otherwise it is
// deferred and blocks its qubits.  The free tile bits are then filled with
// the targets of the earliest deferred gates and the scan is repeated with
// the tile fixed, so that the pass takes every gate that became possible.
std::vector<Sched> schedule(const Group &g, const std::vector<int> &items, int n, int t, int c, int cap,
                            bool earlier_tie)
{
    std::vector<Sched> out;
    if (n <= t) {
        Sched s;
        for (int b = 0; b < n; b++) s.bits.push_back(b);
        if (cap <= 0) {
            s.items = items;
            out.push_back(s);
        } else {
            for (size_t i = 0; i < items.size(); i += cap) {
                s.items.assign(items.begin() + i, items.begin() + std::min(items.size(), i + cap));
                out.push_back(s);
            }
        }
        return out;
    }
    auto pos = [n](int q) { return n - 1 - q; };
    std::vector<int> remaining = items;
    while (!remaining.empty()) {
        std::vector<char> in_tile(n, 0);
        int used = 0;
        for (int b = 0; b < c; b++) in_tile[b] = 1, used++;
        // phase 1: choose bits greedily in gate order
        {
            std::vector<char> blocked(n, 0);
            for (int gi : remaining) {
                int qs[2], ts[2];
                int nq = qubits_of(g, gi, qs), nt = targets(g, gi, ts);
                bool blk = false;
                for (int j = 0; j < nq; j++) blk |= blocked[qs[j]] != 0;
                int need = 0;
                for (int j = 0; j < nt; j++) need += !in_tile[pos(ts[j])];
                if (!blk && used + need <= t) {
                    for (int j = 0; j < nt; j++)
                        if (!in_tile[pos(ts[j])]) in_tile[pos(ts[j])] = 1, used++;
                } else {
                    for (int j = 0; j < nq; j++) blocked[qs[j]] = 1;
                }
            }
        }
        // phase 2: fill free bits with targets of deferred gates, in order
        if (used < t) {
            for (int gi : remaining) {
                int ts[2];
                int nt = targets(g, gi, ts);
                for (int j = 0; j < nt && used < t; j++)
                    if (!in_tile[pos(ts[j])]) in_tile[pos(ts[j])] = 1, used++;
                if (used == t) break;
            }
            for (int b = n - 1; b >= 0 && used < t; b--)
                if (!in_tile[b]) in_tile[b] = 1, used++;
        }
        // phase 3: schedule with the tile fixed -- every gate in order whose
        // target bits are in the tile and whose qubits no earlier deferred
        // gate blocks
        auto place = [&](const std::vector<char> &tile, std::vector<int> *items, std::vector<int> *deferred,
                         int *first_deferred) {
            std::vector<char> blocked(n, 0);
            int count = 0;
            *first_deferred = (int)g.gates.size();
            for (int gi : remaining) {
                int qs[2], ts[2];
                int nq = qubits_of(g, gi, qs), nt = targets(g, gi, ts);
                bool ok = true;
                for (int j = 0; j < nq; j++) ok &= !blocked[qs[j]];
                for (int j = 0; j < nt; j++) ok &= tile[pos(ts[j])] != 0;
                if (ok) {
                    count++;
                    if (items) items->push_back(gi);
                } else {
                    if (*first_deferred == (int)g.gates.size()) *first_deferred = gi;
                    if (deferred) deferred->push_back(gi);
                    for (int j = 0; j < nq; j++) blocked[qs[j]] = 1;
                }
            }
            return count;
        };
        // local search over the tile's free bits: swap one in-tile bit above
        // the low ones for one outside while that places more gates (ties:
        // the first deferred gate comes later, or with earlier_tie earlier),
        // at most kTileSearchSteps swaps
        if (cap <= 0) {
            int fd;
            int best = place(in_tile, nullptr, nullptr, &fd), best_fd = fd;
            for (int step = 0; step < kTileSearchSteps; step++) {
                bool found = false;
                for (int bi = c; bi < n && !found; bi++) {
                    if (!in_tile[bi]) continue;
                    for (int bo = c; bo < n && !found; bo++) {
                        if (in_tile[bo]) continue;
                        in_tile[bi] = 0;
                        in_tile[bo] = 1;
                        const int cnt = place(in_tile, nullptr, nullptr, &fd);
                        if (cnt > best || (cnt == best && (earlier_tie ? fd < best_fd : fd > best_fd))) {
                            best = cnt;
                            best_fd = fd;
                            found = true;
                        } else {
                            in_tile[bi] = 1;
                            in_tile[bo] = 0;
                        }
                    }
                }
                if (!found) break;
            }
        }
        Sched s;
        for (int b = 0; b < n; b++)
            if (in_tile[b]) s.bits.push_back(b);
        std::vector<int> deferred;
        int fd_unused;
        place(in_tile, &s.items, &deferred, &fd_unused);
        if (s.items.empty()) fail(TQ_E_UNSUPPORTED, "planner made no progress");
        if (cap > 0 && (int)s.items.size() > cap) {
            // keep the first `cap` gates; everything else stays in order
            std::vector<char> kept(g.gates.size(), 0);
            s.items.resize(cap);
            for (int gi : s.items) kept[gi] = 1;
            deferred.clear();
            for (int gi : remaining)
                if (!kept[gi]) deferred.push_back(gi);
        }
        out.push_back(std::move(s));
        remaining.swap(deferred);
    }
    return out;
}

// The schedule with the fewest passes of both tie rules of the tile search;
// and for c >= 6 the same with one low bit fewer forced into every tile, which
// frees a tile bit for the search (a pass whose tile holds the bit anyway
// keeps c contiguous low bits, pass_low).  Contiguous runs of 2^5 complex64
// (256 bytes) stream about as fast as runs of 2^6 (gate passes at 24-30
// qubits: within 3%), runs of 2^4 lose 8-15%, so c - 1 stops at 5; and it is
// taken only when it saves at least two passes and a tenth of them, since a
// heavier pass of fp64-bound ops gains little from a sweep fewer (the
// 30-qubit random circuit: 29 -> 22 passes).
std::vector<Sched> schedule_best(const Group &g, const std::vector<int> &items, int n, int t, int c, int cap)
{
    auto best_of_ties = [&](int cc) {
        std::vector<Sched> a = schedule(g, items, n, t, cc, cap, false);
        std::vector<Sched> b = schedule(g, items, n, t, cc, cap, true);
        return b.size() < a.size() ? b : a;
    };
    std::vector<Sched> best = best_of_ties(c);
    if (c - 1 >= 5 && n > t) {
        std::vector<Sched> fewer = best_of_ties(c - 1);
        const size_t save = std::max<size_t>(2, (best.size() + 9) / 10);
        if (fewer.size() + save <= best.size()) best = std::move(fewer);
    }
    return best;
}

// Contiguous low bits of a pass: the run of tile bits from bit 0, at most c.
int pass_low(const std::vector<int> &bits, int c)
{
    int k = 0;
    while (k < c && std::find(bits.begin(), bits.end(), k) != bits.end()) k++;
    return k;
}

TileGeom geom_from_bits(int n, int c, const std::vector<int> &bits)
{
    TileGeom gm{};
    gm.n = n;
    gm.t = (int)bits.size();
    gm.c = std::min(c, n);
    if (gm.t <= gm.c) gm.c = gm.t;
    gm.h = gm.t - gm.c;
    uint64_t tile_mask = 0;
    for (int b : bits) tile_mask |= 1ull << b;
    for (int b = 0; b < gm.c; b++)
        if (!((tile_mask >> b) & 1)) fail(TQ_E_UNSUPPORTED, "tile lacks a low bit");
    int k = 0;
    for (int b : bits)
        if (b >= gm.c) gm.hb[k++] = (uint8_t)b;
    uint64_t all = n >= 64 ? ~0ull : ((1ull << n) - 1);
    gm.fixed_mask = all & ~tile_mask;
    return gm;
}

uint8_t local_of(const TileGeom &gm, int pos)
{
    if (pos < gm.c) return (uint8_t)pos;
    for (int k = 0; k < gm.h; k++)
        if (gm.hb[k] == pos) return (uint8_t)(gm.c + k);
    return kFixed;
}

struct Planner {
    Group &g;
    int32_t alloc(int entries)
    {
        int32_t o = g.mat_block;
        g.mat_block += entries;
        return o;
    }
    int add_task(uint8_t kind, int dim, int storage, int which, const std::vector<Member> &mem)
    {
        BuildTask bt{};
        bt.kind = kind;
        bt.dim = (uint8_t)dim;
        bt.diag = (uint8_t)storage;
        bt.which = (uint8_t)which;
        bt.out = alloc(storage == 1 ? dim : storage == 4 ? 6 : storage >= 2 ? 2 : dim * dim);
        bt.mem_begin = (int32_t)g.members.size();
        bt.mem_count = (int32_t)mem.size();
        for (const auto &m : mem) g.members.push_back(m);
        g.tasks.push_back(bt);
        return (int)g.tasks.size() - 1;
    }
};

// Register stages.  A stage is a set of ops of a pass whose dense
// (non-diagonal) tile bits fit a set R of at most rmax bits (rdense when it
// holds a dense 4x4 or fSim-type op) and that hold at most kMaxStageGrads
// gradient parameters; each thread keeps the 2^|R| amplitudes of one item in
// registers while the stage's ops run.  Diagonal ops and control bits
// outside R read their bit from the item's base index.  Ops commute when
// they act diagonally on every qubit they share, so the ops of a pass are
// reordered within that dependency order to pack them into few stages.
// R is padded with the highest free tile bits, so that the items of
// neighbouring lanes sit at neighbouring LDS addresses.
namespace stages {

std::vector<int> need(const PassOp &op)
{
    std::vector<int> v;
    if (op.kind == K_M1) v.push_back(op.l0);
    if (op.kind == K_M2 || op.kind == K_P2 || op.kind == K_F2) {
        v.push_back(op.l0);
        v.push_back(op.l1);
    }
    return v;
}

bool is_dense(const PassOp &op) { return op.kind == K_M2 || op.kind == K_F2; }

// bits that make an op act alike on all items of a stage when they are
// register bits: also a control bit, and the in-tile bits of a diagonal
std::vector<int> soft(const PassOp &op)
{
    std::vector<int> v = need(op);
    auto add = [&](uint8_t l) {
        if (l != kFixed && std::find(v.begin(), v.end(), (int)l) == v.end()) v.push_back(l);
    };
    if (op.kind == K_M1 && op.ctrl) add(op.l1);
    if (op.kind == K_D1) add(op.l0);
    if (op.kind == K_D2) {
        add(op.l0);
        add(op.l1);
    }
    return v;
}

bool has(const std::vector<int> &bits, int b) { return std::find(bits.begin(), bits.end(), b) != bits.end(); }

// R padded to rs bits with the highest free tile bits, ascending
std::vector<int> padded(std::vector<int> bits, int rs, int t)
{
    for (int b = t - 1; b >= 0 && (int)bits.size() < rs; b--)
        if (!has(bits, b)) bits.push_back(b);
    std::sort(bits.begin(), bits.end());
    return bits;
}

// an op acts alike on all items of a stage with these register bits
bool uniform(const PassOp &op, const std::vector<int> &bits)
{
    for (int b : soft(op))
        if (!has(bits, b)) return false;
    if ((op.kind == K_D1 || op.kind == K_D2) && op.l0 == kFixed) return false;
    if (op.kind == K_D2 && op.l1 == kFixed) return false;
    if (op.kind == K_M1 && op.ctrl && op.l1 == kFixed) return false;
    return true;
}

// fp64-instruction equivalents per amplitude of one op in a register stage
int op_cost(const PassOp &op, int dispatch)
{
    // a diagonal op's entries that are exactly 1 cost nothing in generated
    // kernels (the table-driven ones multiply every entry)
    const bool generated = dispatch == kOpDispatchCostSpec;
    int c = 4;
    if (generated && op.kind == K_D1) c = 2 * (2 - __builtin_popcount(op.hint & 3u));
    if (generated && op.kind == K_D2) c = 4 - __builtin_popcount(op.hint & 15u);
    if (op.kind == K_M1) c = op.ctrl || (op.hint & (kHintReal | kHintRX)) ? 4 : 8;
    if (op.kind == K_M2) c = 16;
    if (op.kind == K_F2) {
        c = (op.hint & kHintRX) ? 4 : 6;
        if (generated) {
            // per four amplitudes: 4 for each |00>, |11> phase that is not 1,
            // and the block: 0 as -i SWAP, 8 in RX form, 16 dense
            const int ph = 4 * (!(op.hint & 1) + !(op.hint & 8));
            const int blk = (op.hint & kHintSwap) ? 2 : (op.hint & kHintRX) ? 8 : 16;
            c = (ph + blk + 3) / 4;
        }
    }
    if (op.kind == K_P2) c = 8;
    return c + dispatch;
}

struct Packing {
    std::vector<int> order;  // ops in stage order
    struct St {
        std::vector<int> bits;  // padded register bits
        int begin, end;         // range in `order`
        bool dense2;            // holds a dense two-qubit op
    };
    std::vector<St> st;
    int cost = 0;
};

// Greedy packing.  commute: use the commutation of diagonal ops (else ops
// sharing any qubit keep their order); soft_first: grow R with the bits that
// make an op uniform, and take uniform ops before per-item ones.
Packing pack(const Pass &ps, int rmax, int rdense, bool commute, bool soft_first, bool forward, int dispatch)
{
    const int t = ps.geom.t;
    const int r = std::min(rmax, t);
    const int rd = std::min(rdense, r);
    const int nops = (int)ps.ops.size();
    std::vector<std::vector<int>> succ(nops);
    std::vector<int> indeg(nops, 0);
    {
        std::map<int, int> last_nd;                  // qubit -> latest op not diagonal on it
        std::map<int, std::vector<int>> diag_since;  // qubit -> ops diagonal on it since then
        for (int k = 0; k < nops; k++) {
            const PassOp &op = ps.ops[k];
            std::vector<std::pair<int, bool>> qs;  // (qubit, op diagonal on it)
            const bool diag = commute && (op.kind == K_D1 || op.kind == K_D2);
            qs.push_back({op.p0, diag});
            if (op.kind == K_M1 && op.ctrl) qs.push_back({op.p1, commute});
            else if (op.kind != K_D1 && op.kind != K_M1) qs.push_back({op.p1, diag});
            std::vector<int> preds;
            auto dep = [&](int pr) {
                if (std::find(preds.begin(), preds.end(), pr) == preds.end()) preds.push_back(pr);
            };
            for (auto &qd : qs) {
                auto it = last_nd.find(qd.first);
                if (it != last_nd.end()) dep(it->second);
                if (qd.second) {
                    diag_since[qd.first].push_back(k);
                } else {
                    for (int pr : diag_since[qd.first]) dep(pr);
                    diag_since[qd.first].clear();
                    last_nd[qd.first] = k;
                }
            }
            for (int pr : preds) succ[pr].push_back(k);
            indeg[k] = (int)preds.size();
        }
    }
    std::set<int> ready;
    for (int k = 0; k < nops; k++)
        if (indeg[k] == 0) ready.insert(k);
    Packing P;
    while (!ready.empty()) {
        std::vector<int> R;
        bool dense = false;
        int ngrad = 0;
        const int begin = (int)P.order.size();
        auto union_with = [&](const std::vector<int> &bits) {
            std::vector<int> u = R;
            for (int b : bits)
                if (!has(u, b)) u.push_back(b);
            return u;
        };
        auto fits = [&](int k, const std::vector<int> &bits, bool dense_now, bool soft_bits) {
            const PassOp &op = ps.ops[k];
            if (ngrad + op.ngrad > kMaxStageGrads) return false;
            for (int b : soft_bits ? soft(op) : need(op))
                if (!has(bits, b)) return false;
            return !((dense_now || is_dense(op)) && (int)bits.size() > rd);
        };
        auto take = [&](bool soft_bits) {
            bool any = false, took = true;
            while (took) {
                took = false;
                for (auto it = ready.begin(); it != ready.end(); ++it) {
                    const int k = *it;
                    if (!fits(k, R, dense, soft_bits)) continue;
                    P.order.push_back(k);
                    ngrad += ps.ops[k].ngrad;
                    dense = dense || is_dense(ps.ops[k]);
                    ready.erase(it);
                    for (int sk : succ[k])
                        if (--indeg[sk] == 0) ready.insert(sk);
                    took = any = true;
                    break;
                }
            }
            return any;
        };
        // grow R by the bits of the ready op that lets the most ready ops fit
        auto grow = [&]() {
            int best = -1, best_score = -1;
            std::vector<int> best_u;
            int considered = 0;
            for (int k : ready) {
                if (++considered > 64) break;
                const PassOp &op = ps.ops[k];
                if (ngrad + op.ngrad > kMaxStageGrads) continue;
                const bool dn = dense || is_dense(op);
                std::vector<int> u = union_with(soft_first ? soft(op) : need(op));
                if ((int)u.size() > (dn ? rd : r)) u = union_with(need(op));
                if ((int)u.size() > (dn ? rd : r) || u.size() == R.size()) continue;
                int score = 0;
                for (int j : ready)
                    if (fits(j, u, dn, soft_first)) score++;
                if (score > best_score) {
                    best = k;
                    best_score = score;
                    best_u = u;
                }
            }
            if (best < 0) return false;
            R = best_u;
            return true;
        };
        for (;;) {
            if (soft_first && take(true)) continue;
            if (!soft_first && take(false)) continue;
            if (grow()) continue;
            if (soft_first && take(false)) continue;
            break;
        }
        if ((int)P.order.size() == begin) fail(TQ_E_UNSUPPORTED, "internal planner error: empty stage");
        Packing::St st{padded(R, dense ? rd : r, t), begin, (int)P.order.size(), dense};
        // modelled cost: one LDS round trip plus the ops, or the dense
        // matrix where the stage can use one
        int ops = 0;
        bool uni = forward;
        for (int i = begin; i < st.end; i++) {
            ops += op_cost(ps.ops[P.order[i]], dispatch);
            uni = uni && uniform(ps.ops[P.order[i]], st.bits);
        }
        const int dense_cost = (4 << (int)st.bits.size()) + (dispatch == kOpDispatchCostSpec ? 2 : 0);
        P.cost += kStageCost + (uni ? std::min(ops, dense_cost) : ops);
        P.st.push_back(st);
    }
    if ((int)P.order.size() != nops) fail(TQ_E_UNSUPPORTED, "internal planner error: op dependency cycle");
    return P;
}

} // namespace stages

void make_stages(Pass &ps, int rmax, int rdense, Group &g, const std::map<int32_t, int> &task_at, bool forward,
                 int dispatch)
{
    const int nops = (int)ps.ops.size();
    ps.stages.clear();
    stages::Packing best;
    bool first = true;
    for (int v = 0; v < 4; v++) {
        stages::Packing P = stages::pack(ps, rmax, rdense, v & 1, v & 2, forward, dispatch);
        if (first || P.cost < best.cost) best = std::move(P);
        first = false;
    }
    std::vector<PassOp> ops(nops);
    for (int k = 0; k < nops; k++) ops[k] = ps.ops[best.order[k]];
    ps.ops = std::move(ops);
    // diagonal ops move past the non-diagonal ops of their stage that act on
    // other qubits (the two commute, and so do their generators), so that a
    // stage's diagonal ops form runs the kernels apply as one diagonal: later
    // in forward stages (a layer's RZ after its RY), earlier in reverse ones
    // (the layer's daggers come in the opposite order)
    auto is_d = [](const PassOp &op) { return op.kind == K_D1 || op.kind == K_D2; };
    auto disjoint = [](const PassOp &a, const PassOp &b) {
        auto qs = [](const PassOp &op, int *q) {
            int n = 0;
            q[n++] = op.p0;
            if (op.kind == K_M2 || op.kind == K_D2 || op.kind == K_P2 || op.kind == K_F2 || (op.kind == K_M1 && op.ctrl))
                q[n++] = op.p1;
            return n;
        };
        int qa[2], qb[2];
        const int na = qs(a, qa), nb = qs(b, qb);
        for (int i = 0; i < na; i++)
            for (int j = 0; j < nb; j++)
                if (qa[i] == qb[j]) return false;
        return true;
    };
    for (const auto &sl : best.st) {
        if (forward) {
            for (int k = sl.end - 2; k >= sl.begin; k--)
                for (int i = k; i + 1 < sl.end && is_d(ps.ops[i]) && !is_d(ps.ops[i + 1]) &&
                                disjoint(ps.ops[i], ps.ops[i + 1]);
                     i++)
                    std::swap(ps.ops[i], ps.ops[i + 1]);
        } else {
            for (int k = sl.begin + 1; k < sl.end; k++)
                for (int i = k; i > sl.begin && is_d(ps.ops[i]) && !is_d(ps.ops[i - 1]) && disjoint(ps.ops[i], ps.ops[i - 1]);
                     i--)
                    std::swap(ps.ops[i], ps.ops[i - 1]);
        }
    }

    for (auto &sl : best.st) {
        const std::vector<int> &bits = sl.bits;
        const int rs = (int)bits.size();
        Stage st{};
        st.r = (uint8_t)rs;
        for (int j = 0; j < rs; j++) st.bits[j] = (uint8_t)bits[j];
        st.op_begin = ps.op_offset + sl.begin;
        st.op_end = ps.op_offset + sl.end;
        for (int k = sl.begin; k < sl.end; k++) {
            PassOp &op = ps.ops[k];
            auto idx = [&](uint8_t l) -> uint8_t {
                for (int j = 0; j < rs; j++)
                    if (l != kFixed && bits[j] == l) return (uint8_t)j;
                return kFixed;
            };
            op.s0 = idx(op.l0);
            op.s1 = idx(op.l1);
            // dense 4x4 ops are stored with their first qubit on the lower
            // register bit: swap the op's qubits and its matrices' qubit order
            if ((op.kind == K_M2 || op.kind == K_F2) && op.s0 > op.s1) {
                std::swap(op.l0, op.l1);
                std::swap(op.p0, op.p1);
                std::swap(op.s0, op.s1);
                std::vector<int32_t> outs{op.mat};
                for (int j = 0; j < op.ngrad; j++) outs.push_back(op.dmat[j]);
                for (int32_t o : outs) {
                    const BuildTask &bt = g.tasks[task_at.at(o)];
                    for (int mi = 0; mi < bt.mem_count; mi++) g.members[bt.mem_begin + mi].swapped ^= 1;
                }
            }
        }
        ps.stages.push_back(st);
    }
}

// A stage is fusable when every op acts alike on all items: its register
// bits, and for controls and diagonals every bit, lie in the stage.
bool stage_fusable(const Pass &ps, const Stage &st)
{
    for (int k = st.op_begin - ps.op_offset; k < st.op_end - ps.op_offset; k++) {
        const PassOp &op = ps.ops[k];
        switch (op.kind) {
        case K_M1:
            if (op.ctrl && op.s1 == kFixed) return false;
            break;
        case K_D1:
            if (op.s0 == kFixed) return false;
            break;
        case K_D2:
            if (op.s0 == kFixed || op.s1 == kFixed) return false;
            break;
        default: break;
        }
    }
    return true;
}

// Dense stage cost (fp64 instructions per amplitude: a 2^r x 2^r complex
// matvec, 4 per entry of a row) against the ops' own costs plus their
// dispatch overhead.
bool dense_pays(const Pass &ps, const Stage &st, int dispatch)
{
    int ops = 0;
    for (int k = st.op_begin - ps.op_offset; k < st.op_end - ps.op_offset; k++)
        ops += stages::op_cost(ps.ops[k], dispatch);
    // a dense stage: 4 per entry of a matrix row, plus (generated kernels)
    // reading its 2^(2r) entries through the scalar cache per item
    return (4 << st.r) + (dispatch == kOpDispatchCostSpec ? 2 : 0) < ops;
}

// Append a pass, split into consecutive passes over the same tile when its
// matrices would not fit the LDS staging area (op k owns the matrix entries
// from its offset up to the next op's).
void push_split(std::vector<Pass> &out, Pass ps)
{
    if (ps.mat_end - ps.mat_begin <= kMaxPassMat) {
        out.push_back(std::move(ps));
        return;
    }
    Pass cur;
    cur.geom = ps.geom;
    cur.product_init = ps.product_init;
    cur.mat_begin = ps.mat_begin;
    for (size_t k = 0; k < ps.ops.size(); k++) {
        const int32_t op_begin = ps.ops[k].mat;
        const int32_t op_end = k + 1 < ps.ops.size() ? ps.ops[k + 1].mat : ps.mat_end;
        if (op_end - cur.mat_begin > kMaxPassMat && !cur.ops.empty()) {
            cur.mat_end = op_begin;
            out.push_back(cur);
            cur.ops.clear();
            cur.mat_begin = op_begin;
            cur.product_init = false;
        }
        cur.ops.push_back(ps.ops[k]);
    }
    cur.mat_end = ps.mat_end;
    out.push_back(std::move(cur));
}

int op_dim(const PassOp &op)
{
    return (op.kind == K_M2 || op.kind == K_D2 || op.kind == K_P2 || op.kind == K_F2) ? 4 : 2;
}

// how the builder stores an op's matrix: 0 dense, 1 diagonal, 2 / 3 the
// pair (a, b) of a I + b XX / a I + b YY
int storage_of(const PassOp &op)
{
    if (op.kind == K_D1 || op.kind == K_D2) return 1;
    if (op.kind == K_P2) return op.ptype == 1 ? 2 : 3;
    if (op.kind == K_F2) return 4;
    return 0;
}

// Structure a gate's matrix has for every parameter value (PassOp::hint):
// the diagonal entries that are exactly 1 (entry index 2 bit(q0) + bit(q1);
// the gates listed are symmetric in their qubits), or exactly X.
uint8_t gate_hint(int op, bool cblock)
{
    switch (op) {
    case OP_Z: case OP_ZPOW: case OP_RZ: return 1;  // diag(1, .) (RZ without its global phase)
    case OP_CZ: case OP_CZPOW: return 1 | 2 | 4;     // diag(1, 1, 1, .)
    case OP_ZZPOW: case OP_RZZ: return 1 | 8;        // diag(1, ., ., 1)
    case OP_X: return kHintX | kHintReal;
    case OP_CNOT: return cblock ? kHintX | kHintReal : 0;
    case OP_RY: case OP_H: return kHintReal;  // real for every angle, and so is dRY/dtheta
    case OP_RX: return kHintRX;               // cos on the diagonal, -i sin off it
    // power gates without their global phase e^{i pi t/2}: cos I - i sin G
    case OP_XPOW: case OP_SQRTX: case OP_XXPOW: case OP_YYPOW: return kHintRX;
    case OP_YPOW: case OP_SQRTY: return kHintReal;
    default: return 0;
    }
}

// The K_F2 hint of one member gate: fSim keeps 1 on |00> and an RX-form
// block; SWAP keeps 1 on |00> and |11>; a diagonal gate keeps its unit
// entries on |00> and |11>, and the block's form when its |01> and |10>
// entries are exactly 1.
uint8_t f2_member_hint(int op)
{
    if (op == OP_FSIM) return 1 | kHintRX;
    if (op == OP_SWAP) return 1 | 8;
    const uint8_t u = gate_hint(op, false) & 0xf;
    return (u & 9) | ((u & 6) == 6 ? kHintRX : 0);
}

// The hint of an op fusing `mem`: entries that are 1 in every member stay 1;
// an X stays X only alone.
uint8_t op_hint(const Group &g, const PassOp &op, const std::vector<Member> &mem)
{
    if (op.kind == K_D1 || op.kind == K_D2) {
        uint8_t h = 0xf;
        for (const Member &m : mem) h &= gate_hint(g.gates[m.gate].op, false) & 0xf;
        return h;
    }
    if (op.kind == K_P2) {  // a I + b P with a real, b imaginary stays so under products
        uint8_t h = kHintRX;
        for (const Member &m : mem) h &= gate_hint(g.gates[m.gate].op, false);
        return h;
    }
    if (op.kind == K_F2) {
        uint8_t h = 1 | 8 | kHintRX;
        for (const Member &m : mem) h &= f2_member_hint(g.gates[m.gate].op);
        return h;
    }
    if (op.kind == K_M1) {
        // a product of real matrices is real, of RX-form matrices RX-form; an
        // X stays X only alone
        uint8_t h = kHintReal | kHintRX;
        for (const Member &m : mem) h &= gate_hint(g.gates[m.gate].op, m.form == FORM_CBLOCK);
        if (mem.size() == 1) h |= gate_hint(g.gates[mem[0].gate].op, mem[0].form == FORM_CBLOCK) & kHintX;
        return h;
    }
    return 0;
}

// Generator terms of gate `opcode` w.r.t. its parameter `which`, in the op
// frame: a controlled gate's op has its target as q0 and its control as q1,
// every other two-qubit op keeps the gate's qubit order (q0 the first).
// Rotations are exp(-i eta P / 2); power gates P^t = exp(-i pi t (P - I) / 2)
// (the phase convention of the program format); fSim(theta, phi) =
// exp(-i theta (XX + YY) / 2) exp(-i phi |11><11|), two commuting factors.
bool gate_generator(int opcode, int which, std::vector<GenTerm> *t)
{
    constexpr double h = 0.5, q = 0.25, hp = M_PI / 2, qp = M_PI / 4;
    t->clear();
    auto add = [&](int x, int z, int ny, double c) { t->push_back(GenTerm{(uint8_t)x, (uint8_t)z, (uint8_t)ny, c}); };
    switch (opcode) {
    case OP_RX: add(1, 0, 0, h); return true;
    case OP_RY: add(1, 1, 1, h); return true;  // Y = i X Z
    case OP_RZ: add(0, 1, 0, h); return true;
    case OP_XPOW: add(1, 0, 0, hp); add(0, 0, 0, -hp); return true;
    case OP_YPOW: add(1, 1, 1, hp); add(0, 0, 0, -hp); return true;
    case OP_ZPOW: add(0, 1, 0, hp); add(0, 0, 0, -hp); return true;
    case OP_XXPOW: add(3, 0, 0, hp); add(0, 0, 0, -hp); return true;
    case OP_YYPOW: add(3, 3, 2, hp); add(0, 0, 0, -hp); return true;  // YY = -XX ZZ
    case OP_ZZPOW: add(0, 3, 0, hp); add(0, 0, 0, -hp); return true;
    case OP_RZZ: add(0, 3, 0, h); return true;
    case OP_CZPOW:  // (pi/2)(CZ - I) = -pi |11><11| = -(pi/4)(I - Z0 - Z1 + Z0 Z1)
        add(0, 0, 0, -qp); add(0, 1, 0, qp); add(0, 2, 0, qp); add(0, 3, 0, -qp);
        return true;
    case OP_CNOTPOW:  // (pi/2)|1><1|_c (X_t - I) = (pi/4)(X_t - I - Z_c X_t + Z_c); t = q0, c = q1
        add(1, 0, 0, qp); add(0, 0, 0, -qp); add(1, 2, 0, -qp); add(0, 2, 0, qp);
        return true;
    case OP_FSIM:
        if (which == 0) {  // (XX + YY) / 2
            add(3, 0, 0, h); add(3, 3, 2, h);
        } else {           // |11><11| = (I - Z0 - Z1 + Z0 Z1) / 4
            add(0, 0, 0, q); add(0, 1, 0, -q); add(0, 2, 0, -q); add(0, 3, 0, q);
        }
        return true;
    default: return false;
    }
}

PassOp base_op(const Group &g, const TileGeom &gm, int gi, int n)
{
    PassOp op{};
    int cls = classify(g.gates[gi].op);
    int q0 = g.gate_q0[gi], q1 = g.gate_q1[gi];
    auto pos = [n](int q) { return n - 1 - q; };
    switch (cls) {
    case C_1D: op.kind = K_D1; break;
    case C_1M: op.kind = K_M1; break;
    case C_CTRL: op.kind = K_M1; break;
    case C_2D: op.kind = K_D2; break;
    case C_2P:
        op.kind = K_P2;
        op.ptype = g.gates[gi].op == OP_XXPOW ? 1 : 2;
        break;
    case C_2F: op.kind = K_F2; break;
    default: op.kind = K_M2; break;
    }
    if (cls == C_CTRL) {  // q0 field = target, q1 field = control
        op.p0 = (uint8_t)pos(q1);
        op.l0 = local_of(gm, op.p0);
        op.p1 = (uint8_t)pos(q0);
        op.l1 = local_of(gm, op.p1);
        op.ctrl = 1;
        op.cval = 1;
    } else {
        op.p0 = (uint8_t)pos(q0);
        op.l0 = local_of(gm, op.p0);
        if (g.gates[gi].nq == 2) {
            op.p1 = (uint8_t)pos(q1);
            op.l1 = local_of(gm, op.p1);
        } else {
            op.p1 = 0;
            op.l1 = kFixed;
        }
    }
    return op;
}

// The global phase the builder leaves out of a gate's matrix (the matrix is
// e^{i phase} times the one built), linear in its parameter: phase = c eta,
// or the constant c.  Rotations about Z and ZZ: e^{-i eta/2}; power gates of
// X, Y, XX and YY: e^{i pi t/2}; sqrt X, sqrt Y and sqrt W: e^{i pi/4}.
bool gate_phase(int op, double *c, bool *constant)
{
    *constant = false;
    switch (op) {
    case OP_RZ: case OP_RZZ: *c = -0.5; return true;
    case OP_XPOW: case OP_YPOW: case OP_XXPOW: case OP_YYPOW: *c = 0.5 * M_PI; return true;
    case OP_SQRTX: case OP_SQRTY: case OP_SQRTW: *c = 0.25 * M_PI; *constant = true; return true;
    default: return false;
    }
}

} // namespace

double gate_left_out_phase(int op, double eta)
{
    double c;
    bool constant;
    if (!gate_phase(op, &c, &constant)) return 0.0;
    return constant ? c : c * eta;
}

namespace {

// A single fSim gate whose (|01>, |10>) block is -i SWAP in every row: theta a
// constant with |cos theta| <= 1e-15 and |sin theta - 1| <= 1e-15 (theta =
// pi/2, the random-circuit coupler): the generated kernels then move the pair
// instead of multiplying it by entries of ~6e-17 and ~1.
bool fsim_swap_block(const Group &g, int gi)
{
    if (g.gates[gi].op != OP_FSIM) return false;
    const int slot = g.gates[gi].slot0;
    if (g.slot_sym[slot] >= 0) return false;
    const size_t rows = g.uniform_slots ? 1 : g.rows.size();
    for (size_t r = 0; r < rows; r++) {
        const double th = g.slot_off[r * (size_t)g.n_slots + slot];
        if (!(std::fabs(std::cos(th)) <= 1e-15 && std::fabs(std::sin(th) - 1.0) <= 1e-15)) return false;
    }
    return true;
}

// Arithmetic per amplitude (fp64 instructions) of a single-qubit op fusing
// `mem` in a generated kernel: diagonal 2 per entry that is not exactly 1,
// dense 4 when real or RX-form, else 8.
int one_qubit_cost(const Group &g, const std::vector<Member> &mem)
{
    bool diag = true;
    for (const Member &m : mem) diag = diag && classify(g.gates[m.gate].op) == C_1D;
    PassOp t{};
    t.kind = diag ? K_D1 : K_M1;
    const uint8_t h = op_hint(g, t, mem);
    if (diag) return 2 * (2 - __builtin_popcount(h & 3u));
    return (h & (kHintReal | kHintRX)) ? 4 : 8;
}

void plan_group(Group &g, const Options &opt, int S)
{
    const int n = g.n;
    Planner P{g};
    const int G = (int)g.gates.size();

    // terms of the row's global phase; the constant ones summed into one
    double phase_const = 0.0;
    for (int gi = 0; gi < G; gi++) {
        double c;
        bool constant;
        if (!gate_phase(g.gates[gi].op, &c, &constant)) continue;
        if (constant) phase_const += c;
        else g.phase_terms.push_back(PhaseTerm{g.gates[gi].slot0, 0, c});
    }
    if (phase_const != 0.0) g.phase_terms.push_back(PhaseTerm{-1, 0, phase_const});

    // Product-state initialisation: the single-qubit gates a qubit sees
    // before its first two-qubit gate act on |0> alone, so the first pass
    // generates the product state instead of reading |0...0> and applying
    // them.
    std::vector<std::vector<int>> absorbed(n);
    std::vector<char> entangled(n, 0), is_absorbed(G, 0);
    for (int gi = 0; gi < G; gi++) {
        if (g.gates[gi].nq == 1 && !entangled[g.gate_q0[gi]]) {
            absorbed[g.gate_q0[gi]].push_back(gi);
            is_absorbed[gi] = 1;
        } else if (g.gates[gi].nq == 2) {
            entangled[g.gate_q0[gi]] = entangled[g.gate_q1[gi]] = 1;
        }
    }
    g.fwd_tasks.begin = (int)g.tasks.size();
    for (int q = 0; q < kMaxQubits; q++) g.init_mat[q] = -1;
    for (int q = 0; q < n; q++) {
        std::vector<Member> mem;
        for (int gi : absorbed[q]) mem.push_back(Member{gi, 0, FORM_FULL, {0, 0}});
        int ti = P.add_task(BT_PRODUCT, 2, 0, 0, mem);
        g.init_mat[q] = g.tasks[ti].out;
    }

    // forward passes
    std::vector<int> fitems;
    for (int gi = 0; gi < G; gi++)
        if (!is_absorbed[gi]) fitems.push_back(gi);
    auto fs = schedule_best(g, fitems, n, opt.tile, opt.low, opt.max_pass_gates);
    if (fs.empty()) {  // nothing beyond the product state: one generating pass
        Sched s;
        for (int b = 0; b < std::min(n, opt.tile); b++) s.bits.push_back(b);
        if (n > opt.tile)
            for (int b = opt.low; (int)s.bits.size() < opt.tile; b++)
                if (std::find(s.bits.begin(), s.bits.end(), b) == s.bits.end()) s.bits.push_back(b);
        std::sort(s.bits.begin(), s.bits.end());
        fs.push_back(s);
    }
    for (size_t pi = 0; pi < fs.size(); pi++) {
        Pass ps;
        ps.geom = geom_from_bits(n, pass_low(fs[pi].bits, opt.low), fs[pi].bits);
        ps.product_init = pi == 0;
        struct OpB {
            PassOp op;
            std::vector<Member> mem;
            int qa, qb;  // qubit set; qb = -1 for one qubit, -2 for a controlled op
        };
        std::vector<OpB> ops;
        std::vector<int> last(n, -1);  // last op touching each qubit
        for (int gi : fs[pi].items) {
            int cls = classify(g.gates[gi].op);
            int q0 = g.gate_q0[gi], q1 = g.gate_q1[gi];
            if (opt.fuse && (cls == C_1D || cls == C_1M)) {
                int o = last[q0];
                const Member mg{gi, 0, FORM_FULL, {0, 0}};
                // generated kernels spend nothing per op, so a product that
                // loses its factors' structure (RY RZ: real and diagonal with
                // a unit entry, dense and complex together) is kept apart when
                // the factors are cheaper one by one
                bool merge = o >= 0 && ops[o].qb == -1 && ops[o].qa == q0;
                if (merge && opt.specialize) {
                    std::vector<Member> both = ops[o].mem;
                    both.push_back(mg);
                    merge = one_qubit_cost(g, both) <= one_qubit_cost(g, ops[o].mem) + one_qubit_cost(g, {mg});
                }
                if (merge) {
                    ops[o].mem.push_back(mg);
                    if (cls == C_1M) ops[o].op.kind = K_M1;
                    continue;
                }
            }
            if (opt.fuse && (cls == C_2D || cls == C_2M || cls == C_2P || cls == C_2F)) {
                int o = last[q0];
                if (o >= 0 && last[q1] == o && ops[o].qb >= 0 &&
                    ((ops[o].qa == q0 && ops[o].qb == q1) || (ops[o].qa == q1 && ops[o].qb == q0))) {
                    ops[o].mem.push_back(Member{gi, (uint8_t)(ops[o].qa != q0), FORM_FULL, {0, 0}});
                    // products of a I + b P with one P keep that form (P^2 = I,
                    // and P is symmetric in its two qubits); anything else is dense
                    const uint8_t pt = g.gates[gi].op == OP_XXPOW ? 1 : 2;
                    const uint8_t k = ops[o].op.kind;
                    if (cls == C_2P && k == K_P2 && ops[o].op.ptype == pt) continue;
                    // diagonal and excitation-preserving gates stay in their classes
                    if (cls == C_2D && k == K_D2) continue;
                    if ((cls == C_2D || cls == C_2F) && (k == K_D2 || k == K_F2)) {
                        ops[o].op.kind = K_F2;
                        continue;
                    }
                    ops[o].op.kind = K_M2;
                    continue;
                }
            }
            OpB ob;
            ob.op = base_op(g, ps.geom, gi, n);
            ob.mem.push_back(Member{gi, 0, (uint8_t)(cls == C_CTRL ? FORM_CBLOCK : FORM_FULL), {0, 0}});
            ob.qa = cls == C_CTRL ? q1 : q0;
            ob.qb = cls == C_CTRL ? -2 : (g.gates[gi].nq == 2 ? q1 : -1);
            int oi = (int)ops.size();
            ops.push_back(std::move(ob));
            last[q0] = oi;
            if (g.gates[gi].nq == 2) last[q1] = oi;
        }
        ps.mat_begin = pi == 0 ? 0 : g.mat_block;
        for (auto &ob : ops) {
            int ti = P.add_task(BT_PRODUCT, op_dim(ob.op), storage_of(ob.op), 0, ob.mem);
            ob.op.mat = g.tasks[ti].out;
            ob.op.hint = op_hint(g, ob.op, ob.mem);
            if (ob.op.kind == K_F2 && ob.mem.size() == 1 && fsim_swap_block(g, ob.mem[0].gate))
                ob.op.hint |= kHintSwap;
            ps.ops.push_back(ob.op);
        }
        ps.mat_end = g.mat_block;
        push_split(g.fwd, std::move(ps));
    }
    g.fwd_tasks.end = (int)g.tasks.size();
    g.fwd_mat_end = g.mat_block;

    // reverse passes: every gate, last first, W^dagger and dW/deta per op;
    // two states share the LDS, so the tile is one bit smaller at most 12
    g.rev_tasks.begin = (int)g.tasks.size();
    std::vector<int> ritems;
    for (int gi = G - 1; gi >= 0; gi--) ritems.push_back(gi);
    int trev = std::min(opt.tile, 12);
    const int crev = std::min(opt.low, trev - 2);
    // (a group without symbolic parameters never runs its reverse passes:
    // one schedule is enough)
    bool symbolic = false;
    for (int gi = 0; gi < G && !symbolic; gi++)
        for (int j = 0; j < g.gates[gi].np; j++) symbolic |= g.slot_sym[g.gates[gi].slot0 + j] >= 0;
    auto rs0 = symbolic ? schedule_best(g, ritems, n, trev, crev, opt.max_pass_gates)
                        : schedule(g, ritems, n, trev, crev, opt.max_pass_gates, false);
    // the reverse kernel keeps per-wave accumulators of every gradient slot of
    // a pass in LDS: split passes that would hold too many
    std::vector<Sched> rs;
    for (auto &s0 : rs0) {
        Sched cur;
        cur.bits = s0.bits;
        int ng = 0;
        for (int gi : s0.items) {
            int k = 0;
            for (int j = 0; j < g.gates[gi].np; j++) k += g.slot_sym[g.gates[gi].slot0 + j] >= 0;
            if (ng + k > kMaxGradPerPass && !cur.items.empty()) {
                rs.push_back(cur);
                cur.items.clear();
                ng = 0;
            }
            cur.items.push_back(gi);
            ng += k;
        }
        if (!cur.items.empty() || rs.empty()) rs.push_back(cur);
    }
    for (auto &s : rs) {
        Pass ps;
        ps.geom = geom_from_bits(n, pass_low(s.bits, crev), s.bits);
        ps.mat_begin = g.mat_block;
        for (int gi : s.items) {
            int cls = classify(g.gates[gi].op);
            PassOp op = base_op(g, ps.geom, gi, n);
            const int dim = op_dim(op), diag = storage_of(op);
            Member m{gi, 0, (uint8_t)(cls == C_CTRL ? FORM_CBLOCK : FORM_FULL), {0, 0}};
            int ti = P.add_task(BT_DAGGER, dim, diag, 0, {m});
            op.mat = g.tasks[ti].out;
            op.hint = op_hint(g, op, {m});  // W^dagger keeps the structure of W
            op.ngrad = 0;
            for (int j = 0; j < g.gates[gi].np; j++) {
                int slot = g.gates[gi].slot0 + j;
                if (g.slot_sym[slot] < 0) continue;
                int di = P.add_task(BT_DERIV, dim, diag, j, {m});
                op.dmat[op.ngrad] = g.tasks[di].out;
                op.gslot[op.ngrad] = g.n_gslots++;
                g.gslot_slot.push_back(slot);
                op.ngrad++;
            }
            ps.ops.push_back(op);
        }
        ps.mat_end = g.mat_block;
        push_split(g.rev, std::move(ps));
    }
    g.rev_tasks.end = (int)g.tasks.size();

    // register stages of every pass
    std::map<int32_t, int> task_at;
    for (int i = 0; i < (int)g.tasks.size(); i++) task_at[g.tasks[i].out] = i;
    int off = 0;
    const int dispatch = opt.specialize ? kOpDispatchCostSpec : kOpDispatchCost;
    for (Pass &ps : g.fwd) {
        ps.op_offset = off;
        // generated tile passes (states too large to run resident) hold
        // four-bit stages, 16 amplitudes per thread in registers: fewer LDS
        // round trips per pass; the precompiled kernels and the resident
        // ones keep kStageBitsFwd, and only stages of at most kStageBitsFwd
        // bits become dense (the stage-matrix builder's limit)
        const int rf = (opt.specialize && n > 12) ? 4 : kStageBitsFwd;
        make_stages(ps, rf, rf, g, task_at, true, dispatch);
        off += (int)ps.ops.size();
        // forward stages whose ops act alike on every item become one dense
        // matrix when that is cheaper than the ops one by one (matrix
        // entries appended to the row block, built after the op matrices)
        for (Stage &st : ps.stages) {
            if (st.r > kStageBitsFwd || !stage_fusable(ps, st) || !dense_pays(ps, st, dispatch)) continue;
            st.dense = 1;
            st.mat = g.mat_block;
            g.mat_block += 1 << (2 * st.r);
            g.dense_stages.push_back({(int)(&ps - g.fwd.data()), (int)(&st - ps.stages.data())});
        }
    }
    off = 0;
    for (Pass &ps : g.rev) {
        ps.op_offset = off;
        make_stages(ps, rev_stage_bits(n, opt), kRevDense2Bits, g, task_at, false, dispatch);
        off += (int)ps.ops.size();
    }

    // every dense op must find its target bits in the tile
    for (const std::vector<Pass> *pv : {&g.fwd, &g.rev})
        for (const Pass &ps : *pv)
            for (const PassOp &op : ps.ops) {
                bool ok = true;
                if (op.kind == K_M1) ok = op.l0 < ps.geom.t && (!op.ctrl || op.l1 == kFixed || op.l1 < ps.geom.t);
                if (op.kind == K_M2 || op.kind == K_P2 || op.kind == K_F2)
                    ok = op.l0 < ps.geom.t && op.l1 < ps.geom.t && op.l0 != op.l1;
                if (op.kind == K_D1 || op.kind == K_D2) ok = op.p0 < n && (op.kind == K_D1 || op.p1 < n);
                if (!ok) fail(TQ_E_UNSUPPORTED, "internal planner error: op outside its tile");
            }

    // symbol -> gradient slots
    g.sym_gslot_begin.assign(S + 1, 0);
    for (int gs = 0; gs < g.n_gslots; gs++) g.sym_gslot_begin[g.slot_sym[g.gslot_slot[gs]] + 1]++;
    for (int s = 0; s < S; s++) g.sym_gslot_begin[s + 1] += g.sym_gslot_begin[s];
    g.sym_gslots.assign(g.n_gslots, 0);
    std::vector<int> fill(g.sym_gslot_begin.begin(), g.sym_gslot_begin.end() - 1);
    for (int gs = 0; gs < g.n_gslots; gs++) g.sym_gslots[fill[g.slot_sym[g.gslot_slot[gs]]]++] = gs;
}

} // namespace

bool op_generator(const Group &g, const PassOp &op, int j, std::vector<GenTerm> *terms)
{
    if (j >= op.ngrad) return false;
    for (int k = g.rev_tasks.begin; k < g.rev_tasks.end; k++) {
        const BuildTask &bt = g.tasks[k];
        if (bt.kind != BT_DERIV || bt.out != op.dmat[j] || bt.mem_count != 1) continue;
        return gate_generator(g.gates[g.members[bt.mem_begin].gate].op, bt.which, terms);
    }
    return false;
}

TileGeom expectation_geometry(int n, int t, int c, const std::vector<uint64_t> &xmasks)
{
    std::vector<int> bits;
    if (n <= t) {
        for (int b = 0; b < n; b++) bits.push_back(b);
        return geom_from_bits(n, c, bits);
    }
    std::vector<int> count(n, 0);
    for (uint64_t x : xmasks)
        for (int b = 0; b < n; b++)
            if ((x >> b) & 1) count[b]++;
    for (int b = 0; b < c; b++) bits.push_back(b);
    std::vector<int> rest;
    for (int b = c; b < n; b++) rest.push_back(b);
    std::stable_sort(rest.begin(), rest.end(), [&](int a, int b) { return count[a] > count[b]; });
    for (int i = 0; (int)bits.size() < t; i++) bits.push_back(rest[i]);
    std::sort(bits.begin(), bits.end());
    return geom_from_bits(n, c, bits);
}

PauliTables pauli_tables(int n, int t, int c, int K, const std::vector<std::vector<TermDev>> &per_row, bool uniform)
{
    PauliTables pt;
    std::vector<uint64_t> xs;
    for (size_t r = 0; r < per_row.size() && (r == 0 || !uniform); r++)
        for (const TermDev &td : per_row[r]) xs.push_back(td.x);
    pt.geom = expectation_geometry(n, std::min(n, t), std::min(c, std::min(n, t)), xs);
    const TileGeom &gm = pt.geom;
    auto local = [&](uint64_t m) {
        uint32_t v = 0;
        for (int k = 0; k < gm.c; k++)
            if ((m >> k) & 1) v |= 1u << k;
        for (int k = 0; k < gm.h; k++)
            if ((m >> gm.hb[k]) & 1) v |= 1u << (gm.c + k);
        return v;
    };
    struct Item {
        int chunk;
        uint64_t xF;
        uint32_t xT;
        int k;
        uint32_t u;
        PTerm term;
    };
    const int nchunk = (K + kPauliChunk - 1) / kPauliChunk;
    pt.row_begin.assign(per_row.size(), 0);
    pt.row_count.assign(per_row.size(), nchunk);
    for (size_t r = 0; r < per_row.size(); r++) {
        if (uniform && r > 0) {
            pt.row_begin[r] = pt.row_begin[0];
            continue;
        }
        std::vector<Item> items;
        items.reserve(per_row[r].size());
        for (const TermDev &td : per_row[r]) {
            Item it{};
            it.chunk = td.k / kPauliChunk;
            it.k = td.k;
            it.xF = td.x & gm.fixed_mask;
            it.xT = local(td.x);
            const uint32_t zT = local(td.z);
            it.u = zT >> 8;
            // c' = c i^{ny} chi_z(x): real for even ny, imaginary for odd ny
            const int ny = td.ny & 3;
            double v = td.coeff;
            if (__builtin_popcountll(td.z & td.x) & 1) v = -v;
            if (ny >= 2) v = -v;
            it.term = PTerm{td.z & gm.fixed_mask, zT & 0xffu, (uint32_t)(ny & 1), v};
            if (it.xF) pt.partner = true;
            items.push_back(it);
        }
        std::stable_sort(items.begin(), items.end(), [](const Item &a, const Item &b) {
            if (a.chunk != b.chunk) return a.chunk < b.chunk;
            if (a.xF != b.xF) return a.xF < b.xF;
            if (a.xT != b.xT) return a.xT < b.xT;
            if (a.k != b.k) return a.k < b.k;
            return a.u < b.u;
        });
        pt.row_begin[r] = (int32_t)pt.chunks.size();
        size_t i = 0;
        for (int ci = 0; ci < nchunk; ci++) {
            PChunk ch{};
            ch.k0 = ci * kPauliChunk;
            ch.nk = std::min(kPauliChunk, K - ch.k0);
            ch.xf_begin = (int32_t)pt.xfg.size();
            while (i < items.size() && items[i].chunk == ci) {
                PXfGroup xf{};
                xf.xF = items[i].xF;
                xf.x_begin = (int32_t)pt.xg.size();
                while (i < items.size() && items[i].chunk == ci && items[i].xF == xf.xF) {
                    PXGroup xg{};
                    xg.xT = items[i].xT;
                    xg.kk = items[i].k - ch.k0;
                    xg.u_begin = (int32_t)pt.us.size();
                    const int k = items[i].k;
                    while (i < items.size() && items[i].chunk == ci && items[i].xF == xf.xF && items[i].xT == xg.xT &&
                           items[i].k == k) {
                        PUSub us{};
                        us.u = items[i].u;
                        us.t_begin = (int32_t)pt.terms.size();
                        while (i < items.size() && items[i].chunk == ci && items[i].xF == xf.xF &&
                               items[i].xT == xg.xT && items[i].k == k && items[i].u == us.u) {
                            xg.flags |= items[i].term.im ? 2u : 1u;
                            pt.terms.push_back(items[i].term);
                            i++;
                        }
                        us.t_end = (int32_t)pt.terms.size();
                        pt.us.push_back(us);
                    }
                    xg.u_end = (int32_t)pt.us.size();
                    pt.xg.push_back(xg);
                }
                xf.x_end = (int32_t)pt.xg.size();
                pt.xfg.push_back(xf);
            }
            ch.xf_end = (int32_t)pt.xfg.size();
            pt.chunks.push_back(ch);
        }
    }
    return pt;
}

// Covers tried besides the greedy one when planning the passes of an
// observable set (each a greedy fill of the tile bits in a shuffled term
// order); the plan with the fewest passes is kept.
constexpr int kCoverTrials = 256;

bool pauli_spec_plan(int n, int t, int c, const std::vector<TermDev> &terms, std::vector<PauliPass> *passes)
{
    passes->clear();
    const int h = t - c;
    const uint64_t low = (1ull << c) - 1;
    std::vector<uint64_t> xs;  // the terms' X bits above the low ones
    for (const TermDev &td : terms) {
        if (__builtin_popcountll(td.x & ~low) > h) return false;
        xs.push_back(td.x & ~low);
    }
    // greedy: grow the set S of high tile bits one X mask at a time, the one
    // that keeps S within h bits and covers the most terms left
    std::vector<uint64_t> cover;
    {
        std::vector<uint64_t> left = xs;
        while (!left.empty()) {
            uint64_t S = 0;
            for (;;) {
                uint64_t best = 0;
                size_t best_cov = 0;
                int best_size = 0;
                for (uint64_t x : left) {
                    const uint64_t U = S | x;
                    if (U == S || __builtin_popcountll(U) > h) continue;
                    size_t cov = 0;
                    for (uint64_t o : left) cov += (o & ~U) == 0;
                    const int size = __builtin_popcountll(U);
                    if (cov > best_cov || (cov == best_cov && size < best_size)) {
                        best = U;
                        best_cov = cov;
                        best_size = size;
                    }
                }
                if (!best) break;
                S = best;
            }
            cover.push_back(S);
            std::vector<uint64_t> rest;
            for (uint64_t x : left)
                if (x & ~S) rest.push_back(x);
            left.swap(rest);
        }
    }
    // shuffled fills (a fixed counter-based shuffle per trial): keep one
    // with fewer passes
    for (int trial = 0; trial < kCoverTrials && cover.size() > 1; trial++) {
        std::vector<uint64_t> left = xs, cv;
        uint64_t st = 0x9E3779B97F4A7C15ull * (uint64_t)(trial + 1);
        while (!left.empty() && cv.size() + 1 < cover.size()) {
            for (size_t i = left.size(); i > 1; i--) {  // Fisher-Yates with SplitMix64 draws
                st += 0x9E3779B97F4A7C15ull;
                uint64_t z = st;
                z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
                z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
                z ^= z >> 31;
                std::swap(left[i - 1], left[z % i]);
            }
            uint64_t S = 0;
            for (uint64_t x : left)
                if (__builtin_popcountll(S | x) <= h) S |= x;
            cv.push_back(S);
            std::vector<uint64_t> rest;
            for (uint64_t x : left)
                if (x & ~S) rest.push_back(x);
            left.swap(rest);
        }
        if (left.empty() && cv.size() < cover.size()) cover = cv;
    }
    // the passes: each tile the low bits, the cover's bits and filler bits;
    // each term in the first pass whose tile holds its X bits
    std::vector<const TermDev *> left;
    for (const TermDev &td : terms) left.push_back(&td);
    for (uint64_t S : cover) {
        std::vector<int> bits;
        for (int b = 0; b < c; b++) bits.push_back(b);
        for (int b = c; b < n; b++)
            if ((S >> b) & 1) bits.push_back(b);
        for (int b = c; b < n && (int)bits.size() < t; b++)
            if (!((S >> b) & 1)) bits.push_back(b);
        std::sort(bits.begin(), bits.end());
        PauliPass ps;
        ps.geom = geom_from_bits(n, c, bits);
        std::vector<const TermDev *> rest;
        for (const TermDev *td : left) {
            if (((td->x & ~low) & ~S) == 0)
                ps.terms.push_back(SpecTerm{td->k, td->x, td->z, td->ny, td->coeff});
            else
                rest.push_back(td);
        }
        if (!ps.terms.empty()) passes->push_back(std::move(ps));
        left.swap(rest);
    }
    return left.empty();
}

DiagTables diag_tables(const std::vector<std::vector<TermDev>> &per_row, bool uniform)
{
    DiagTables dt;
    struct Item {
        int k;
        uint32_t v, zT;
        uint64_t zB;
        double c;
    };
    dt.row_begin.assign(per_row.size(), 0);
    dt.row_count.assign(per_row.size(), 0);
    for (size_t r = 0; r < per_row.size(); r++) {
        if (uniform && r > 0) {
            dt.row_begin[r] = dt.row_begin[0];
            dt.row_count[r] = dt.row_count[0];
            continue;
        }
        std::vector<Item> items;
        for (const TermDev &td : per_row[r]) {
            if (td.x) fail(TQ_E_INVALID, "internal error: diagonal tables for a term with X or Y factors");
            const uint64_t z = td.z;
            items.push_back(Item{td.k, (uint32_t)((z & 1) | (((z >> 9) & 7) << 1)), (uint32_t)((z >> 1) & 0xff),
                                 z >> kDiagBlockBits, td.coeff});
        }
        std::stable_sort(items.begin(), items.end(), [](const Item &a, const Item &b) {
            if (a.k != b.k) return a.k < b.k;
            if (a.v != b.v) return a.v < b.v;
            if (a.zT != b.zT) return a.zT < b.zT;
            return a.zB < b.zB;
        });
        dt.row_begin[r] = (int32_t)dt.chunks.size();
        DChunk ch{};
        ch.c_begin = (int32_t)dt.classes.size();
        auto close_chunk = [&]() {
            ch.c_end = (int32_t)dt.classes.size();
            if (ch.c_end > ch.c_begin) {
                ch.k_lo = dt.classes[ch.c_begin].k;
                ch.k_hi = dt.classes[ch.c_end - 1].k;
                dt.amax = std::max(dt.amax, ch.c_end - ch.c_begin);
                dt.chunks.push_back(ch);
            }
            ch.c_begin = ch.c_end;
        };
        for (size_t i = 0; i < items.size();) {
            if ((int)dt.classes.size() - ch.c_begin == kDiagClassMax) close_chunk();
            DClass cl{};
            cl.k = items[i].k;
            cl.v = items[i].v;
            cl.zT = items[i].zT;
            cl.t_begin = (int32_t)dt.terms.size();
            for (; i < items.size() && items[i].k == cl.k && items[i].v == cl.v && items[i].zT == cl.zT; i++) {
                // equal block masks share one weight term
                if (dt.terms.size() > (size_t)cl.t_begin && dt.terms.back().zB == items[i].zB)
                    dt.terms.back().c += items[i].c;
                else
                    dt.terms.push_back(DTerm{items[i].zB, items[i].c});
            }
            cl.t_end = (int32_t)dt.terms.size();
            dt.classes.push_back(cl);
        }
        close_chunk();
        dt.row_count[r] = (int32_t)dt.chunks.size() - dt.row_begin[r];
    }
    return dt;
}

// exp(-i eta P) for a Pauli string P (Sec. "Quantum Neural Networks",
// eqs. Pauli_decomp and cs_decomp), read from the blob after its header
// (nq = the string's weight w, np = 1: w qubits, the parameter, w Pauli
// codes) and written as gates of the fixed table, which the planner fuses:
// each X factor turned into Z by H on both sides, each Y by RX(pi/2) before
// and RX(-pi/2) after (RX(t)^dag Z RX(t) = cos t Z + sin t Y); the Z string
// by RZZ(2 eta) for weight two, and for more by a CNOT ladder that gathers
// the parity of the first w - 1 qubits into the (w-1)-th, RZZ(2 eta) with
// the last, and the ladder undone.  Weight one is RX, RY or RZ(2 eta)
// itself; weight zero is the global phase exp(-i eta) = RZ(2 eta)
// ZPOW(-2 eta / pi) on qubit 0.
// The parameter keeps its symbol: the emitted rotations scale it by 2 (or
// -2/pi), so the chain rule sums their gradients back onto the symbol.
template <class Emit>
void lower_pauli_exp(Reader &r, const HGate &head, int n, int32_t S, uint32_t b, uint32_t i, Emit &&emit)
{
    const std::string where = "circuit " + std::to_string(b) + " gate " + std::to_string(i);
    const int w = head.nq;
    if (head.np != 1) fail(TQ_E_INVALID, where + ": a Pauli exponential takes one parameter");
    if (w > n) fail(TQ_E_INVALID, where + ": Pauli string longer than the circuit");
    std::vector<uint32_t> qs(w);
    for (int j = 0; j < w; j++) {
        qs[j] = r.get<uint32_t>();
        if (!r.bad && qs[j] >= (uint32_t)n) fail(TQ_E_INVALID, where + ": qubit out of range");
        for (int k = 0; k < j; k++)
            if (qs[k] == qs[j]) fail(TQ_E_INVALID, where + ": repeated qubit");
    }
    const int32_t sym = r.get<int32_t>();
    const double scale = r.get<double>(), offset = r.get<double>();
    if (!r.bad && (sym < -1 || sym >= S)) fail(TQ_E_INVALID, where + ": symbol column out of range");
    std::vector<uint8_t> ps(w);
    for (int j = 0; j < w; j++) {
        ps[j] = r.get<uint8_t>();
        if (!r.bad && (ps[j] < 1 || ps[j] > 3)) fail(TQ_E_INVALID, where + ": Pauli code must be 1 (X), 2 (Y) or 3 (Z)");
    }
    if (r.bad) fail(TQ_E_INVALID, "program blob: truncated gate");
    auto gate = [](int op, uint32_t q0, uint32_t q1 = 0) {
        HGate h{};
        h.op = (uint16_t)op;
        int nq, np;
        op_shape(op, nq, np);
        h.nq = (uint8_t)nq;
        h.np = (uint8_t)np;
        h.q[0] = q0;
        h.q[1] = q1;
        return h;
    };
    auto param = [&](HGate h, double f) {  // the exponential's parameter times f
        h.sym[0] = sym;
        h.scale[0] = f * scale;
        h.offset[0] = f * offset;
        h.mult = f;
        return h;
    };
    auto constant = [](HGate h, double v) {
        h.sym[0] = -1;
        h.offset[0] = v;
        return h;
    };
    if (w == 0) {
        if (n == 0) return;  // no qubit to carry the phase: a circuit without amplitudes to scale
        emit(param(gate(OP_RZ, 0), 2.0));
        emit(param(gate(OP_ZPOW, 0), -2.0 / M_PI));
        return;
    }
    auto basis = [&](bool before) {
        for (int j = 0; j < w; j++) {
            if (ps[j] == 1) emit(gate(OP_H, qs[j]));
            else if (ps[j] == 2) emit(constant(gate(OP_RX, qs[j]), before ? M_PI / 2 : -M_PI / 2));
        }
    };
    if (w == 1) {  // exp(-i eta X) = RX(2 eta), likewise Y and Z: no basis change
        emit(param(gate(ps[0] == 1 ? OP_RX : ps[0] == 2 ? OP_RY : OP_RZ, qs[0]), 2.0));
        return;
    }
    basis(true);
    for (int j = 0; j + 2 < w; j++) emit(gate(OP_CNOT, qs[j], qs[j + 1]));
    emit(param(gate(OP_RZZ, qs[w - 2], qs[w - 1]), 2.0));
    for (int j = w - 3; j >= 0; j--) emit(gate(OP_CNOT, qs[j], qs[j + 1]));
    basis(false);
}

bool shift_rule(int op, int param, double *delta, double *factor)
{
    switch (op) {
    case OP_RX: case OP_RY: case OP_RZ: case OP_RZZ:
        // exp(-i eta G / 2), G^2 = I: eigenvalues +-1/2, gap 1
        *delta = M_PI / 2;
        *factor = 0.5;
        return true;
    case OP_XPOW: case OP_YPOW: case OP_ZPOW: case OP_CZPOW: case OP_CNOTPOW: case OP_XXPOW: case OP_YYPOW:
    case OP_ZZPOW:
        // G^t = e^{i pi t / 2} exp(-i (pi t / 2) G): gap pi in t
        *delta = 0.5;
        *factor = M_PI / 2;
        return true;
    case OP_PAULIEXP:
        // exp(-i eta P): eigenvalues +-1, gap 2 (the rule as the paper prints it)
        *delta = M_PI / 4;
        *factor = 1.0;
        return true;
    case OP_FSIM:
        if (param != 1) return false;  // theta: (XX + YY) / 2 has eigenvalues -1, 0, 1
        // phi: exp(-i phi |11><11|), gap 1
        *delta = M_PI / 2;
        *factor = 0.5;
        return true;
    default:
        return false;
    }
}

std::unique_ptr<ProgramData> parse_program(const void *blob, size_t nbytes, const Options &opt)
{
    if (!blob) fail(TQ_E_INVALID, "program blob is NULL");
    Reader r{(const uint8_t *)blob, (const uint8_t *)blob + nbytes};
    if (nbytes < 16 || std::memcmp(blob, "TQP1", 4) != 0) fail(TQ_E_INVALID, "program blob: bad magic");
    r.p += 4;
    uint32_t ver = r.get<uint32_t>(), B = r.get<uint32_t>(), S = r.get<uint32_t>();
    if (ver != 1) fail(TQ_E_INVALID, "program blob: unsupported version");
    if (B > (1u << 24) || S > (1u << 24)) fail(TQ_E_INVALID, "program blob: batch or symbol count too large");
    auto pd = std::make_unique<ProgramData>();
    pd->B = (int)B;
    pd->S = (int)S;
    pd->opt = opt;
    pd->circuits.resize(B);
    // Each circuit is parsed into one reused scratch list; only the first
    // circuit of a structure keeps its gates (in its group), the others add
    // their scales and offsets to that group's parameter tables.
    std::vector<HGate> gates;
    std::map<std::string, int> key_to_group;
    std::string key;
    for (uint32_t b = 0; b < B; b++) {
        uint32_t n = r.get<uint32_t>(), ng = r.get<uint32_t>();
        if (r.bad) fail(TQ_E_INVALID, "program blob: truncated circuit header");
        if (n > (uint32_t)kMaxQubits)
            fail(TQ_E_UNSUPPORTED, "circuit " + std::to_string(b) + " has more than 32 qubits");
        if (ng > (1u << 24)) fail(TQ_E_INVALID, "program blob: gate count too large");
        HCircuit &c = pd->circuits[b];
        c.n = (int)n;
        pd->nmax = std::max(pd->nmax, (int)n);
        // m: gates of the circuit after lowering (a Pauli-string exponential
        // becomes several gates)
        size_t m = 0;
        auto emit = [&](const HGate &h) {
            if (m == gates.size()) gates.push_back(h);
            else gates[m] = h;
            m++;
        };
        HGate g{};
        for (uint32_t i = 0; i < ng; i++) {
            g.op = r.get<uint16_t>();
            g.nq = r.get<uint8_t>();
            g.np = r.get<uint8_t>();
            g.q[0] = g.q[1] = 0;
            for (int j = 0; j < 3; j++) {
                g.sym[j] = 0;
                g.scale[j] = g.offset[j] = 0.0;
            }
            if (r.bad) fail(TQ_E_INVALID, "program blob: truncated gate");
            if (g.op == OP_PAULIEXP) {
                lower_pauli_exp(r, g, (int)n, (int32_t)S, b, i, [&](HGate h) {
                    h.origin = (int32_t)i;
                    h.blob_op = OP_PAULIEXP;
                    emit(h);
                });
                continue;
            }
            int enq, enp;
            if (!op_shape(g.op, enq, enp))
                fail(TQ_E_UNSUPPORTED, "circuit " + std::to_string(b) + " gate " + std::to_string(i) +
                                           ": unknown opcode " + std::to_string(g.op));
            if (enq != g.nq || enp != g.np)
                fail(TQ_E_INVALID, "circuit " + std::to_string(b) + " gate " + std::to_string(i) +
                                       ": qubit/parameter count does not match the opcode");
            for (int j = 0; j < g.nq; j++) {
                g.q[j] = r.get<uint32_t>();
                if (!r.bad && g.q[j] >= n)
                    fail(TQ_E_INVALID, "circuit " + std::to_string(b) + " gate " + std::to_string(i) +
                                           ": qubit out of range");
            }
            if (g.nq == 2 && g.q[0] == g.q[1])
                fail(TQ_E_INVALID, "circuit " + std::to_string(b) + " gate " + std::to_string(i) +
                                       ": repeated qubit");
            for (int j = 0; j < g.np; j++) {
                g.sym[j] = r.get<int32_t>();
                g.scale[j] = r.get<double>();
                g.offset[j] = r.get<double>();
                if (!r.bad && (g.sym[j] < -1 || g.sym[j] >= (int32_t)S))
                    fail(TQ_E_INVALID, "circuit " + std::to_string(b) + " gate " + std::to_string(i) +
                                           ": symbol column out of range");
            }
            if (g.op == OP_PCHAN && !r.bad) {  // constant probabilities >= 0, summing to <= 1
                double tot = 0.0;
                for (int j = 0; j < 3; j++) {
                    if (g.sym[j] != -1 || !(g.offset[j] >= 0.0))
                        fail(TQ_E_INVALID, "circuit " + std::to_string(b) + " gate " + std::to_string(i) +
                                               ": channel probabilities must be constants >= 0");
                    tot += g.offset[j];
                }
                if (!(tot <= 1.0))
                    fail(TQ_E_INVALID, "circuit " + std::to_string(b) + " gate " + std::to_string(i) +
                                           ": channel probabilities sum above 1");
            }
            const int nm = g.op == OP_MATRIX1 ? 8 : g.op == OP_MATRIX2 ? 32 : 0;
            for (int j = 0; j < nm; j++) g.mat[j] = r.get<double>();
            if (nm)
                for (int j = nm; j < 32; j++) g.mat[j] = 0.0;
            if (r.bad) fail(TQ_E_INVALID, "program blob: truncated gate");
            g.origin = (int32_t)i;
            g.blob_op = g.op;
            g.mult = 1.0;
            emit(g);
        }
        if (m > (size_t)1 << 24) fail(TQ_E_INVALID, "program blob: gate count too large");
        ng = (uint32_t)m;
        // structure dedupe: same qubit count, opcodes, qubits, symbol wiring
        // and explicit matrices; scales and offsets may differ per row
        key.clear();
        key.append((const char *)&c.n, sizeof c.n);
        for (uint32_t i = 0; i < ng; i++) {
            const HGate &g = gates[i];
            key.append((const char *)&g.op, 2);
            key.append((const char *)g.q, 8);
            key.append((const char *)g.sym, sizeof g.sym);
            key.append((const char *)&g.origin, sizeof g.origin);
            if (g.op == OP_MATRIX1 || g.op == OP_MATRIX2)
                key.append((const char *)g.mat, sizeof(double) * (g.op == OP_MATRIX1 ? 8 : 32));
        }
        auto it = key_to_group.find(key);
        Group *grp;
        if (it == key_to_group.end()) {
            key_to_group.emplace(key, (int)pd->groups.size());
            pd->groups.push_back(std::make_unique<Group>());
            grp = pd->groups.back().get();
            grp->n = c.n;
            int nchan = 0;
            std::vector<int32_t> occ_origin;  // blob gate of each occurrence
            for (uint32_t i = 0; i < ng; i++) {
                const HGate &g = gates[i];
                GateDev gd{};
                gd.op = g.op;
                gd.nq = g.nq;
                gd.np = g.np;
                gd.slot0 = grp->n_slots;
                gd.explicit_ = -1;
                gd.chan = g.op == OP_PCHAN ? nchan++ : -1;
                if (g.op == OP_MATRIX1 || g.op == OP_MATRIX2) {
                    gd.explicit_ = (int32_t)(grp->explicit_mats.size() / 32);
                    grp->explicit_mats.insert(grp->explicit_mats.end(), g.mat, g.mat + 32);
                }
                for (int j = 0; j < g.np; j++) {
                    if (g.sym[j] >= 0) {
                        // a blob gate's parameter: lowered gates of one
                        // exponential share it (parameter 0)
                        const int bj = g.blob_op == OP_PAULIEXP ? 0 : j;
                        auto &oc = grp->occurrences;
                        if (!oc.empty() && oc.back().slot[1] < 0 && g.blob_op == OP_PAULIEXP &&
                            oc.back().blob_op == OP_PAULIEXP && occ_origin.back() == g.origin) {
                            oc.back().slot[1] = grp->n_slots + j;
                            oc.back().mult[1] = g.mult;
                        } else {
                            oc.push_back(Occurrence{{grp->n_slots + j, -1}, {g.mult, 0.0}, g.sym[j], g.blob_op,
                                                    (uint8_t)bj});
                            occ_origin.push_back(g.origin);
                        }
                    }
                    grp->slot_sym.push_back(g.sym[j]);
                }
                grp->n_slots += g.np;
                grp->gates.push_back(gd);
                grp->gate_q0.push_back((int32_t)g.q[0]);
                grp->gate_q1.push_back(g.nq == 2 ? (int32_t)g.q[1] : -1);
            }
        } else {
            grp = pd->groups[it->second].get();
        }
        grp->rows.push_back((int32_t)b);
        for (uint32_t i = 0; i < ng; i++)
            for (int j = 0; j < gates[i].np; j++) {
                grp->slot_scale.push_back(gates[i].scale[j]);
                grp->slot_off.push_back(gates[i].offset[j]);
            }
    }
    if (r.p != r.end) fail(TQ_E_INVALID, "program blob: trailing bytes");

    for (auto &gp : pd->groups) {
        Group &g = *gp;
        // rows that share every scale and offset keep one table row
        bool uni = true;
        size_t ns = (size_t)g.n_slots;
        for (size_t r = 1; r < g.rows.size() && uni; r++)
            uni = std::equal(g.slot_scale.begin(), g.slot_scale.begin() + ns, g.slot_scale.begin() + r * ns) &&
                  std::equal(g.slot_off.begin(), g.slot_off.begin() + ns, g.slot_off.begin() + r * ns);
        g.uniform_slots = uni;
        if (uni) {
            g.slot_scale.resize(ns);
            g.slot_off.resize(ns);
        }
        plan_group(g, opt, (int)S);
    }
    return pd;
}

std::unique_ptr<ObsData> parse_observables(const void *blob, size_t nbytes)
{
    if (!blob) fail(TQ_E_INVALID, "observable blob is NULL");
    Reader r{(const uint8_t *)blob, (const uint8_t *)blob + nbytes};
    if (nbytes < 16 || std::memcmp(blob, "TQO1", 4) != 0) fail(TQ_E_INVALID, "observable blob: bad magic");
    r.p += 4;
    uint32_t ver = r.get<uint32_t>(), B = r.get<uint32_t>(), K = r.get<uint32_t>();
    if (ver != 1) fail(TQ_E_INVALID, "observable blob: unsupported version");
    if ((uint64_t)B * K > (1u << 26)) fail(TQ_E_INVALID, "observable blob: too many sums");
    auto od = std::make_unique<ObsData>();
    od->B = (int)B;
    od->K = (int)K;
    od->sums.resize((size_t)B * K);
    for (auto &sum : od->sums) {
        uint32_t T = r.get<uint32_t>();
        if (r.bad || T > (1u << 24)) fail(TQ_E_INVALID, "observable blob: bad term count");
        sum.resize(T);
        for (auto &term : sum) {
            term.coeff = r.get<double>();
            uint32_t nf = r.get<uint32_t>();
            if (r.bad || nf > (uint32_t)kMaxQubits) fail(TQ_E_INVALID, "observable blob: bad factor count");
            uint64_t seen = 0;
            for (uint32_t f = 0; f < nf; f++) {
                uint32_t q = r.get<uint32_t>();
                uint8_t p = r.get<uint8_t>();
                if (r.bad) fail(TQ_E_INVALID, "observable blob: truncated term");
                if (p < 1 || p > 3) fail(TQ_E_INVALID, "observable blob: Pauli code must be 1, 2 or 3");
                if (q >= (uint32_t)kMaxQubits) fail(TQ_E_INVALID, "observable blob: qubit out of range");
                if ((seen >> q) & 1) fail(TQ_E_INVALID, "observable blob: qubit repeated within a term");
                seen |= 1ull << q;
                term.factors.emplace_back(q, p);
            }
        }
    }
    if (r.bad) fail(TQ_E_INVALID, "observable blob: truncated");
    if (r.p != r.end) fail(TQ_E_INVALID, "observable blob: trailing bytes");
    return od;
}

} // namespace tq
