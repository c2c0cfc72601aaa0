// tq_abi.cpp -- the extern "C" entry points of libtq: validation, lazy
// device upload of the plan, workspace management and the launch sequence of
// each call.  Every call validates on the host first and then only enqueues
// work on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <iomanip>
#include <map>
#include <sstream>
#include <cstring>
#include <memory>
#include <string>
#include <vector>

#include "../../include/tq.h"
#include "jit.h"
#include "kernels.h"
#include "program.h"

using namespace tq;

namespace {

thread_local std::string g_err;

[[noreturn]] void fail(int status, const std::string &m) { throw Error{status, m}; }

void hip_check(hipError_t e, const char *what)
{
    if (e != hipSuccess) fail(TQ_E_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

// A device allocation owned by a handle, grown on demand.
struct DevBuf {
    void *p = nullptr;
    size_t bytes = 0;
    void *ensure(size_t n)
    {
        if (n <= bytes && p) return p;
        release();
        if (n == 0) n = 256;
        if (hipMalloc(&p, n) != hipSuccess) {
            (void)hipGetLastError();
            p = nullptr;
            bytes = 0;
            fail(TQ_E_NOMEM, "device allocation of " + std::to_string(n) + " bytes failed");
        }
        bytes = n;
        return p;
    }
    void release()
    {
        if (p) (void)hipFree(p);
        p = nullptr;
        bytes = 0;
    }
};

template <class T> T *upload(DevBuf &buf, const std::vector<T> &v)
{
    size_t n = std::max<size_t>(v.size() * sizeof(T), 16);
    T *d = static_cast<T *>(buf.ensure(n));
    if (!v.empty()) hip_check(hipMemcpy(d, v.data(), v.size() * sizeof(T), hipMemcpyHostToDevice), "hipMemcpy");
    return d;
}

std::atomic<uint64_t> g_obs_counter{1};

int wg_for(int nrows, int tiles_log2)
{
    // enough workgroups to cover the chip several times, never more than the tiles
    int64_t tiles = (int64_t)1 << tiles_log2;
    int64_t want = std::max<int64_t>(1, 4096 / std::max(nrows, 1));
    return (int)std::min<int64_t>(tiles, want);
}

struct ObsGroupDev {
    TileGeom geom;
    int tmax = 0;
    DevBuf terms, begin, count;  // TermDev tables (resident kernel)
    // tables of the tile Pauli kernel
    TileGeom pgeom;
    bool partner = false;
    DevBuf chunks, cbegin, ccount, xfg, xg, us, pterms;
    // tables of the diagonal Pauli kernel (all terms Z-only, n >= kDiagBlockBits)
    bool diag = false;
    int damax = 0;
    DevBuf dchunks, dcbegin, dccount, dclasses, dterms;
    // passes and source of the kernels specialised for the observable set
    // (specialize = 1, every row the same terms, tiles that hold every X mask)
    // sets of at most 16 observables, each with passes of its own
    struct SpecSet {
        int k0 = 0, kc = 0;  // observables [k0, k0 + kc)
        std::vector<PauliPass> passes;
        std::string src;
        SpecMemo memo;
    };
    std::vector<SpecSet> spec_sets;
    // passes and source of the kernels computing phi = g H psi for a single
    // observable the same on every row (specialize = 1)
    std::vector<PauliPass> phi_passes;
    std::string phi_src;
    SpecMemo phi_memo;
    void release()
    {
        for (DevBuf *b : {&terms, &begin, &count, &chunks, &cbegin, &ccount, &xfg, &xg, &us, &pterms, &dchunks,
                          &dcbegin, &dccount, &dclasses, &dterms})
            b->release();
    }
};

// Largest observable (terms) whose phi = g H psi kernels are generated, and
// largest observable set (terms over all its observables) whose expectation
// kernels are.
constexpr size_t kMaxPhiTerms = 1024;
constexpr size_t kMaxSpecTerms = 1024;
// observables per set of generated expectation passes: up to 16 keep
// register accumulators (one set); more are split into sets of up to 200
// with per-wave sums in LDS (8 waves x 200 doubles beside a 2^13-amplitude
// tile still leave two workgroups per CU); and the most terms (over all
// observables) whose passes are generated
constexpr int kSpecSetObs = 16;
constexpr int kSpecSetObsLds = 200;
constexpr size_t kMaxSpecTermsAll = 4096;

// Tile size of the Pauli kernel (log2 amplitudes): 2048 amplitudes, eight
// per thread.
constexpr int kPauliTile = 11;

struct GroupDev {
    DevBuf rows, ident, gates, slot_sym, scale, off, explicit_, tasks, members, fwd_ops, rev_ops, sym_begin,
        sym_gslots, gslot_slot, fwd_stages, rev_stages, dense_list, phase_terms;
    std::vector<int> fwd_op_off, rev_op_off, fwd_stage_off, rev_stage_off;
    int n_fwd_stages = 0, n_rev_stages = 0, n_dense = 0;
    size_t psi_off = 0;  // amplitude offset of this group's rows in the state workspaces
    size_t mat_off = 0;  // offset in the matrix workspace
    // specialised kernels of the group: the resident kernel, the tile passes
    SpecMemo res_memo, pass_memo;
    // the batched shift rules: per kind (0 parameter shift, 1 central
    // differences) the moves of the derived rows, their pairs and the CSR
    // symbol -> pairs; the parameter-shift rows' shot-counter bases
    bool x_ready[2] = {false, false};
    int x_period[2] = {0, 0};
    int x_max_list[2] = {0, 0};  // the longest task list of a move
    DevBuf x_shift[2], x_pair_slot[2], x_pair_coef[2], x_sym_begin[2], x_sym_pairs[2], x_ebase, x_list_begin[2],
        x_list[2], x_phase_full[2], x_phase_begin[2], x_phase_list[2];
    void release_x()
    {
        for (int k = 0; k < 2; k++)
            for (DevBuf *b : {&x_shift[k], &x_pair_slot[k], &x_pair_coef[k], &x_sym_begin[k], &x_sym_pairs[k],
                              &x_list_begin[k], &x_list[k], &x_phase_full[k], &x_phase_begin[k], &x_phase_list[k]})
                b->release();
        x_ebase.release();
    }
};

} // namespace

struct tq_observables_s {
    std::unique_ptr<ObsData> od;
    // Sampled expectations: the non-identity terms as observables of their
    // own with coefficient 1 (row b's observable j is its j-th non-identity
    // term over (k, t); Kt the most any row has), and the shot tables on the
    // device `dev` (one table row when every row has the same terms).
    std::unique_ptr<ObsData> terms;
    int Kt = 0;
    bool uniform = true;
    int dev = -1;
    DevBuf slot_k, slot_t, obs_begin, term_slot, term_coeff;
    int64_t term_stride = 0;
    ~tq_observables_s()
    {
        for (DevBuf *b : {&slot_k, &slot_t, &obs_begin, &term_slot, &term_coeff}) b->release();
    }
};

struct tq_program_s {
    std::unique_ptr<ProgramData> pd;
    int device = -1;
    std::vector<std::unique_ptr<GroupDev>> gdev;
    DevBuf psi, phi, mats, partial, gpart, levels;
    // workspaces of the derived rows (batched shift rules) and of the
    // sampled expectations
    DevBuf xpsi, xmats, xout, xident, xtab[kRowGatherArrays], xterm, xcounts;
    int xident_n = 0;
    size_t psi_total = 0, mat_total = 0;
    uint64_t obs_id = 0;
    std::vector<std::unique_ptr<ObsGroupDev>> obs_dev;
    // tables of the observable sets used before the current one (most
    // recent last), kept so that calls alternating between a few sets do
    // not rebuild them
    std::vector<std::pair<uint64_t, std::vector<std::unique_ptr<ObsGroupDev>>>> obs_kept;
    uint64_t noise_seed = 0;  // seed of the channels' per-row draws

    ~tq_program_s()
    {
        for (auto &g : gdev) {
            g->release_x();
            for (DevBuf *b : {&g->rows, &g->ident, &g->gates, &g->slot_sym, &g->scale, &g->off, &g->explicit_,
                              &g->tasks, &g->members, &g->fwd_ops, &g->rev_ops, &g->sym_begin, &g->sym_gslots,
                              &g->gslot_slot, &g->fwd_stages, &g->rev_stages, &g->dense_list, &g->phase_terms})
                b->release();
        }
        for (auto &o : obs_dev) o->release();
        for (auto &k : obs_kept)
            for (auto &o : k.second) o->release();
        for (DevBuf *b : {&psi, &phi, &mats, &partial, &gpart, &levels, &xpsi, &xmats, &xout, &xident, &xterm,
                          &xcounts})
            b->release();
        for (DevBuf &b : xtab) b.release();
    }
};

namespace {

template <class F> tq_status guarded(F &&f)
{
    try {
        f();
        g_err.clear();
        return TQ_OK;
    } catch (const Error &e) {
        g_err = e.msg;
        return (tq_status)e.status;
    } catch (const std::bad_alloc &) {
        g_err = "host allocation failed";
        return TQ_E_NOMEM;
    } catch (...) {
        g_err = "internal error";
        return TQ_E_DEVICE;
    }
}

// Upload the plan to the current device on first use.
void ensure_device(tq_program p)
{
    int dev = -1;
    hip_check(hipGetDevice(&dev), "hipGetDevice");
    if (p->device >= 0) {
        if (dev != p->device) fail(TQ_E_INVALID, "program was first used on another device");
        return;
    }
    ProgramData &pd = *p->pd;
    size_t psi_total = 0, mat_total = 0;
    for (auto &gp : pd.groups) {
        const Group &g = *gp;
        auto gd = std::make_unique<GroupDev>();
        upload(gd->rows, g.rows);
        std::vector<int32_t> ident(g.rows.size());
        for (size_t i = 0; i < ident.size(); i++) ident[i] = (int32_t)i;
        upload(gd->ident, ident);
        upload(gd->gates, g.gates);
        upload(gd->slot_sym, g.slot_sym);
        upload(gd->scale, g.slot_scale);
        upload(gd->off, g.slot_off);
        upload(gd->explicit_, g.explicit_mats);
        upload(gd->tasks, g.tasks);
        upload(gd->members, g.members);
        upload(gd->phase_terms, g.phase_terms);
        std::vector<PassOp> fo, ro;
        for (const Pass &ps : g.fwd) {
            gd->fwd_op_off.push_back((int)fo.size());
            fo.insert(fo.end(), ps.ops.begin(), ps.ops.end());
        }
        for (const Pass &ps : g.rev) {
            gd->rev_op_off.push_back((int)ro.size());
            ro.insert(ro.end(), ps.ops.begin(), ps.ops.end());
        }
        upload(gd->fwd_ops, fo);
        upload(gd->rev_ops, ro);
        std::vector<Stage> fs, rs;
        for (const Pass &ps : g.fwd) {
            gd->fwd_stage_off.push_back((int)fs.size());
            fs.insert(fs.end(), ps.stages.begin(), ps.stages.end());
        }
        for (const Pass &ps : g.rev) {
            gd->rev_stage_off.push_back((int)rs.size());
            rs.insert(rs.end(), ps.stages.begin(), ps.stages.end());
        }
        gd->n_fwd_stages = (int)fs.size();
        gd->n_rev_stages = (int)rs.size();
        upload(gd->fwd_stages, fs);
        upload(gd->rev_stages, rs);
        std::vector<int32_t> dl;
        for (auto &d : g.dense_stages) dl.push_back(gd->fwd_stage_off[d.first] + d.second);
        gd->n_dense = (int)dl.size();
        upload(gd->dense_list, dl);
        upload(gd->sym_begin, g.sym_gslot_begin);
        upload(gd->sym_gslots, g.sym_gslots);
        upload(gd->gslot_slot, g.gslot_slot);
        gd->psi_off = psi_total;
        // keep every group's rows 512-byte aligned for the vector tile loads
        psi_total += ((g.rows.size() << g.n) + 63) & ~(size_t)63;
        gd->mat_off = mat_total;
        mat_total += g.rows.size() * (size_t)std::max(g.mat_block, 1);
        p->gdev.push_back(std::move(gd));
    }
    p->psi_total = psi_total;
    p->mat_total = mat_total;
    p->device = dev;
}

float2 *psi_ws(tq_program p) { return (float2 *)p->psi.ensure(p->psi_total * sizeof(float2)); }
float2 *phi_ws(tq_program p) { return (float2 *)p->phi.ensure(p->psi_total * sizeof(float2)); }
double2 *mat_ws(tq_program p) { return (double2 *)p->mats.ensure(p->mat_total * sizeof(double2)); }

// The rows one launch sequence over a group runs.  Plain calls run the
// group's own rows (own_rows).  The batched shift rules run derived rows:
// launch row r is row begin + r of the group's expansion, a copy of group row
// (begin + r) / period with the parameter moves of shift[(begin + r) % period],
// its matrices in a workspace of its own, its state at row r of the state
// array and its outputs at row r of the output array.
struct RunRows {
    int n = 0;
    int64_t begin = 0;
    int period = 0;                      // 0: the group's own rows
    const ShiftDev *shift = nullptr;
    double eps = 0.0;                    // central differences: the symbol moves are +-eps
    // derived rows built from their source rows' matrices (x_src): copied,
    // then only the tasks of each move's list built again
    const double2 *x_src = nullptr;
    const int32_t *list_begin = nullptr, *task_list = nullptr;
    const int32_t *phase_full = nullptr, *phase_begin = nullptr, *phase_list = nullptr;
    int max_list = 0;
    double2 *mats = nullptr;
    const int32_t *ident = nullptr;      // 0 .. n-1 (state rows of the workspaces)
    const int32_t *out_rows = nullptr;   // output row of each launch row
    // observable tables of each launch row (NULL: the group's own, by group row)
    const int32_t *term_begin = nullptr, *term_count = nullptr, *cbegin = nullptr, *ccount = nullptr,
                  *dcbegin = nullptr, *dccount = nullptr;
};

RunRows own_rows(tq_program p, size_t gi)
{
    RunRows r;
    r.n = (int)p->pd->groups[gi]->rows.size();
    r.mats = mat_ws(p) + p->gdev[gi]->mat_off;
    r.ident = (const int32_t *)p->gdev[gi]->ident.p;
    r.out_rows = (const int32_t *)p->gdev[gi]->rows.p;
    return r;
}

template <class T> const T *or_own(const int32_t *derived, const DevBuf &own)
{
    return derived ? derived : (const T *)own.p;
}

// Symbol resolution + fused matrices for the task range [begin, end).
void build_mats(tq_program p, size_t gi, const float *theta, int begin, int end, hipStream_t s, const RunRows &rr)
{
    const Group &g = *p->pd->groups[gi];
    GroupDev &gd = *p->gdev[gi];
    BuildArgs a{};
    a.tasks = (const BuildTask *)gd.tasks.p;
    a.task_begin = begin;
    a.task_end = end;
    a.members = (const Member *)gd.members.p;
    a.gates = (const GateDev *)gd.gates.p;
    a.slot_sym = (const int32_t *)gd.slot_sym.p;
    a.slot_scale = (const double *)gd.scale.p;
    a.slot_off = (const double *)gd.off.p;
    a.uniform = g.uniform_slots;
    a.n_slots = g.n_slots;
    a.explicit_mats = (const double *)gd.explicit_.p;
    a.theta = theta;
    a.S = p->pd->S;
    a.rows = (const int32_t *)gd.rows.p;
    a.mats = rr.mats;
    a.mat_stride = std::max(g.mat_block, 1);
    a.x_begin = rr.begin;
    a.x_period = rr.period;
    a.x_shift = rr.shift;
    a.x_eps = rr.eps;
    a.x_src = rr.x_src;
    a.x_copy = g.fwd_mat_end;
    a.list_begin = rr.list_begin;
    a.task_list = rr.task_list;
    a.phase_full = rr.phase_full;
    a.phase_begin = rr.phase_begin;
    a.phase_list = rr.phase_list;
    // the first qubit's product-init matrix (built by the range's first
    // task) carries the row's global phase
    const bool init = g.n > 0 && begin == g.fwd_tasks.begin && end > begin && !g.phase_terms.empty();
    a.phase_out = init ? g.init_mat[0] : -1;
    a.n_phase = (int32_t)g.phase_terms.size();
    a.phase_terms = (const PhaseTerm *)gd.phase_terms.p;
    a.noise_seed = p->noise_seed;
    if (rr.x_src) {
        if (begin != g.fwd_tasks.begin || end != g.fwd_tasks.end)
            fail(TQ_E_INVALID, "derived rows build the forward matrices only");
        hip_check(launch_build_derived(a, rr.n, rr.max_list, s), "derived matrix build launch");
    } else {
        hip_check(launch_build(a, rr.n, s), "matrix build launch");
    }
    if (begin <= g.fwd_tasks.begin && end >= g.fwd_tasks.end && gd.n_dense > 0) {
        // dense forward stages, from the op matrices just built
        StageBuildArgs sb{};
        sb.stages = (const Stage *)gd.fwd_stages.p;
        sb.list = (const int32_t *)gd.dense_list.p;
        sb.nlist = gd.n_dense;
        sb.ops = (const PassOp *)gd.fwd_ops.p;
        sb.mats = a.mats;
        sb.mat_stride = a.mat_stride;
        hip_check(launch_build_stage(sb, rr.n, s), "stage matrix build launch");
    }
}

// Forward passes of group gi into `state` (row r of the group at
// srows[r] * row_stride).
void forward(tq_program p, size_t gi, float2 *state, int64_t row_stride, const int32_t *srows, hipStream_t s,
             const RunRows &rr)
{
    const Group &g = *p->pd->groups[gi];
    GroupDev &gd = *p->gdev[gi];
    const int nrows = rr.n;
    for (size_t pi = 0; pi < g.fwd.size(); pi++) {
        const Pass &ps = g.fwd[pi];
        PassArgs a{};
        a.state = state;
        a.row_stride = row_stride;
        a.rows = srows;
        a.mats = rr.mats;
        a.mat_stride = std::max(g.mat_block, 1);
        a.ops = (const PassOp *)gd.fwd_ops.p;
        a.stages = (const Stage *)gd.fwd_stages.p + gd.fwd_stage_off[pi];
        a.nstages = (int)ps.stages.size();
        a.g = ps.geom;
        a.tiles_log2 = g.n - ps.geom.t;
        a.wg_per_row = wg_for(nrows, a.tiles_log2);
        a.product_init = ps.product_init;
        for (int q = 0; q < kMaxQubits; q++) a.init_mat[q] = g.init_mat[q];
        a.mat_begin = ps.mat_begin;
        a.mat_end = ps.mat_end;
        if (p->pd->opt.specialize) {
            std::string log;
            const hipError_t e = launch_pass_spec(g, (int)pi, a, nrows, s, &log, &gd.pass_memo);
            if (e == hipErrorInvalidSource) fail(TQ_E_DEVICE, log);
            hip_check(e, "specialised pass launch");
            continue;
        }
        hip_check(launch_pass(a, nrows, s), "pass launch");
    }
}

void check_obs_fit(tq_program p, tq_observables o)
{
    const ProgramData &pd = *p->pd;
    const ObsData &od = *o->od;
    if (od.B != pd.B) fail(TQ_E_INVALID, "observables batch size differs from the program's");
    for (int b = 0; b < pd.B; b++)
        for (int k = 0; k < od.K; k++)
            for (const HTerm &t : od.sums[(size_t)b * od.K + k])
                for (auto &f : t.factors)
                    if ((int)f.first >= pd.circuits[b].n)
                        fail(TQ_E_INVALID, "observable (" + std::to_string(b) + ", " + std::to_string(k) +
                                               ") acts on a qubit the circuit does not have");
}

// Per-group term tables of an observables handle, in the group's
// expectation tile geometry.
constexpr size_t kObsKept = 3;

void ensure_obs(tq_program p, const ObsData &od)
{
    if (p->obs_id == od.id) return;
    for (size_t i = 0; i < p->obs_kept.size(); i++)
        if (p->obs_kept[i].first == od.id) {
            auto tables = std::move(p->obs_kept[i].second);
            p->obs_kept.erase(p->obs_kept.begin() + i);
            if (p->obs_id) p->obs_kept.emplace_back(p->obs_id, std::move(p->obs_dev));
            p->obs_dev = std::move(tables);
            p->obs_id = od.id;
            return;
        }
    const ProgramData &pd = *p->pd;
    std::vector<std::unique_ptr<ObsGroupDev>> out;
    for (auto &gp : pd.groups) {
        const Group &g = *gp;
        const int n = g.n;
        std::vector<std::vector<TermDev>> per_row(g.rows.size());
        std::vector<uint64_t> xs;
        for (size_t r = 0; r < g.rows.size(); r++) {
            int b = g.rows[r];
            for (int k = 0; k < od.K; k++)
                for (const HTerm &t : od.sums[(size_t)b * od.K + k]) {
                    TermDev td{};
                    for (auto &f : t.factors) {
                        uint64_t bit = 1ull << (n - 1 - (int)f.first);
                        if (f.second == 1 || f.second == 2) td.x |= bit;
                        if (f.second == 2 || f.second == 3) td.z |= bit;
                        if (f.second == 2) td.ny++;
                    }
                    td.k = k;
                    td.coeff = t.coeff;
                    per_row[r].push_back(td);
                    xs.push_back(td.x);
                }
        }
        auto og = std::make_unique<ObsGroupDev>();
        og->geom = expectation_geometry(n, std::min(p->pd->opt.tile, 12), std::min(p->pd->opt.low, 10), xs);
        const TileGeom &gm = og->geom;
        auto local_mask = [&](uint64_t m) {
            uint32_t r = 0;
            for (int k = 0; k < gm.c; k++)
                if ((m >> k) & 1) r |= 1u << k;
            for (int k = 0; k < gm.h; k++)
                if ((m >> gm.hb[k]) & 1) r |= 1u << (gm.c + k);
            return r;
        };
        bool uniform = true;
        for (auto &row : per_row) {
            for (auto &td : row) {
                td.xout = td.x & gm.fixed_mask;
                td.xl = local_mask(td.x);
                td.zl = local_mask(td.z);
            }
        }
        for (size_t r = 1; r < per_row.size() && uniform; r++)
            uniform = per_row[r].size() == per_row[0].size() &&
                      std::memcmp(per_row[r].data(), per_row[0].data(), per_row[0].size() * sizeof(TermDev)) == 0;
        std::vector<TermDev> flat;
        std::vector<int32_t> begin(g.rows.size()), count(g.rows.size());
        for (size_t r = 0; r < per_row.size(); r++) {
            if (uniform && r > 0) {
                begin[r] = 0;
                count[r] = (int32_t)per_row[0].size();
                continue;
            }
            begin[r] = (int32_t)flat.size();
            count[r] = (int32_t)per_row[r].size();
            flat.insert(flat.end(), per_row[r].begin(), per_row[r].end());
            og->tmax = std::max(og->tmax, count[r]);
        }
        upload(og->terms, flat);
        upload(og->begin, begin);
        upload(og->count, count);
        PauliTables pt = pauli_tables(n, std::min(p->pd->opt.tile, kPauliTile), p->pd->opt.low, od.K, per_row, uniform);
        og->pgeom = pt.geom;
        og->partner = pt.partner;
        upload(og->chunks, pt.chunks);
        upload(og->cbegin, pt.row_begin);
        upload(og->ccount, pt.row_count);
        upload(og->xfg, pt.xfg);
        upload(og->xg, pt.xg);
        upload(og->us, pt.us);
        upload(og->pterms, pt.terms);
        bool diag = n >= kDiagBlockBits;
        for (auto &row : per_row)
            for (auto &td : row) diag = diag && td.x == 0;
        size_t nterms = 0;
        for (auto &row : per_row) nterms = std::max(nterms, row.size());
        if (!diag && p->pd->opt.specialize && uniform && nterms <= kMaxSpecTermsAll) {
            // observables in sets (at most 16 with one register accumulator
            // each, else up to 200 summed per wave in LDS), each set's terms in
            // passes over tiles of 2^12 or 2^13 amplitudes (16 per thread)
            // with runs of 2^5 or 2^6 contiguous amplitudes: the fewest
            // passes weighted by what a pass costs (measured on 2^24..2^30
            // amplitudes: a 2^13 tile streams ~15-20% slower than a 2^12 one,
            // 2^14 tiles and runs of 2^4 much slower)
            bool ok = true;
            const int per_set = od.K <= kSpecSetObs ? kSpecSetObs : kSpecSetObsLds;
            for (int k0 = 0; k0 < od.K && ok; k0 += per_set) {
                ObsGroupDev::SpecSet set;
                set.k0 = k0;
                set.kc = std::min(per_set, od.K - k0);
                std::vector<TermDev> terms;
                for (const TermDev &td : per_row[0])
                    if (td.k >= k0 && td.k < k0 + set.kc) {
                        terms.push_back(td);
                        terms.back().k -= k0;
                    }
                if (terms.size() > kMaxSpecTerms) ok = false;
                double best = 0;
                for (int t = 12; t <= 13 && t < n && ok; t++)
                    for (int c = 6; c >= 5; c--) {
                        std::vector<PauliPass> pp;
                        if (!pauli_spec_plan(n, t, c, terms, &pp)) continue;
                        const double cost = pp.size() * (1.0 + 0.2 * (t - 12)) * (1.0 + 0.05 * (6 - c));
                        if (set.passes.empty() || cost < best) {
                            best = cost;
                            set.passes = std::move(pp);
                        }
                    }
                if (set.passes.empty()) ok = false;
                if (!ok) break;
                set.src = pauli_spec_source(set.passes, set.kc);
                og->spec_sets.push_back(std::move(set));
            }
            if (!ok) og->spec_sets.clear();
        }
        // (states of at most 12 qubits run resident: their phi is formed on chip)
        if (p->pd->opt.specialize && uniform && od.K == 1 && nterms > 0 && nterms <= kMaxPhiTerms && n > 12) {
            // the fewest passes (each reads psi and updates phi), smaller
            // tiles and longer runs on ties
            for (int t = 12; t <= 13 && t < n; t++)
                for (int c = 6; c >= 5; c--) {
                    std::vector<PauliPass> pp;
                    if (!pauli_spec_plan(n, t, c, per_row[0], &pp)) continue;
                    if (og->phi_passes.empty() || pp.size() < og->phi_passes.size()) og->phi_passes = std::move(pp);
                }
            if (!og->phi_passes.empty()) og->phi_src = hphi_spec_source(og->phi_passes);
        }
        if (diag) {
            DiagTables dt = diag_tables(per_row, uniform);
            og->diag = true;
            og->damax = dt.amax;
            upload(og->dchunks, dt.chunks);
            upload(og->dcbegin, dt.row_begin);
            upload(og->dccount, dt.row_count);
            upload(og->dclasses, dt.classes);
            upload(og->dterms, dt.terms);
        }
        out.push_back(std::move(og));
    }
    if (p->obs_id) {
        p->obs_kept.emplace_back(p->obs_id, std::move(p->obs_dev));
        if (p->obs_kept.size() > kObsKept) {
            for (auto &old : p->obs_kept.front().second) old->release();
            p->obs_kept.erase(p->obs_kept.begin());
        }
    }
    p->obs_dev = std::move(out);
    p->obs_id = od.id;
}

// Expectations of Z-only Pauli sums over group gi's rows (n >= 12), streamed
// from HBM by the diagonal kernel.
void diag_group(tq_program p, size_t gi, const float2 *psi, int K, float *out, hipStream_t s, const RunRows &rr)
{
    const Group &g = *p->pd->groups[gi];
    ObsGroupDev &og = *p->obs_dev[gi];
    const int nrows = rr.n;
    DiagArgs a{};
    a.psi = psi;
    a.row_stride = (int64_t)1 << g.n;
    a.rows = rr.ident;
    a.chunks = (const DChunk *)og.dchunks.p;
    a.row_chunk_begin = or_own<int32_t>(rr.dcbegin, og.dcbegin);
    a.row_chunk_count = or_own<int32_t>(rr.dccount, og.dccount);
    a.classes = (const DClass *)og.dclasses.p;
    a.terms = (const DTerm *)og.dterms.p;
    a.blocks_log2 = g.n - kDiagBlockBits;
    // one round of workgroups over the device (as many as fit at once), each
    // sweeping many blocks: no partial last round
    const int64_t nblk = (int64_t)1 << a.blocks_log2;
    int fit = pauli_diag_slots(og.damax, std::min(K, 1024));
    if (fit <= 0) fit = 2048;
    a.wg_per_row = (int)std::max<int64_t>(1, std::min<int64_t>(nblk, fit / nrows));
    const int64_t slots = (int64_t)nrows * a.wg_per_row;
    const int kmax = (int)std::max<int64_t>(1, std::min<int64_t>(1024, ((int64_t)32 << 20) / slots));
    for (int k0 = 0; k0 < K; k0 += kmax) {
        a.k_begin = k0;
        a.k_count = std::min(kmax, K - k0);
        a.partial = (double *)p->partial.ensure(sizeof(double) * (size_t)slots * a.k_count);
        hip_check(launch_pauli_diag(a, nrows, og.damax, s), "diagonal Pauli kernel launch");
        PauliReduceArgs r{};
        r.rows = rr.out_rows;
        r.partial = a.partial;
        r.wg_per_row = a.wg_per_row;
        r.K = K;
        r.k_begin = k0;
        r.k_count = a.k_count;
        r.out = out;
        hip_check(launch_pauli_reduce(r, nrows, s), "Pauli reduce launch");
    }
}

// Expectations of an observable set the same on every row of group gi, by
// the kernels specialised for it: one state read per pass of the plan.
void spec_pauli_group(tq_program p, size_t gi, const float2 *psi, int K, float *out, hipStream_t s,
                      const RunRows &rr)
{
    const Group &g = *p->pd->groups[gi];
    ObsGroupDev &og = *p->obs_dev[gi];
    const int nrows = rr.n;
    std::string log;
    // launch shapes of every set first: the partial workspace is sized once
    // for the largest (no reallocation while an earlier set's work runs)
    std::vector<int> wg(og.spec_sets.size());
    size_t need = 1;
    for (size_t si = 0; si < og.spec_sets.size(); si++) {
        ObsGroupDev::SpecSet &set = og.spec_sets[si];
        int fit = pauli_spec_slots(set.src, set.passes[0].geom, set.kc, &log, &set.memo);
        if (fit <= 0) {
            if (!log.empty()) fail(TQ_E_DEVICE, log);
            fit = 2048;
        }
        const int64_t ntiles = (int64_t)1 << (g.n - set.passes[0].geom.t);
        // sets beyond kSpecSetObs observables: one workgroup per tile (their
        // kernels store per-tile sums)
        wg[si] = set.kc > kSpecSetObs ? (int)ntiles : (int)std::max<int64_t>(1, std::min<int64_t>(ntiles, fit / nrows));
        need = std::max(need, (size_t)nrows * set.passes.size() * wg[si] * set.kc);
    }
    double *partial = (double *)p->partial.ensure(sizeof(double) * need);
    for (size_t si = 0; si < og.spec_sets.size(); si++) {
        ObsGroupDev::SpecSet &set = og.spec_sets[si];
        const int npass = (int)set.passes.size();
        PauliSpecArgs a{};
        a.psi = psi;
        a.row_stride = (int64_t)1 << g.n;
        a.rows = rr.ident;
        a.wg_per_row = wg[si];
        a.npass = npass;
        a.k_count = set.kc;
        a.partial = partial;
        for (int pi = 0; pi < npass; pi++) {
            a.g = set.passes[pi].geom;
            a.pass = pi;
            const hipError_t e = launch_pauli_spec(set.src, pi, a, nrows, s, &log, &set.memo);
            if (e == hipErrorInvalidSource) fail(TQ_E_DEVICE, log);
            hip_check(e, "specialised Pauli launch");
        }
        PauliReduceArgs r{};
        r.rows = rr.out_rows;
        r.partial = partial;
        r.wg_per_row = npass * a.wg_per_row;  // the passes' workgroups side by side
        r.K = K;
        r.k_begin = set.k0;
        r.k_count = set.kc;
        r.out = out;
        hip_check(launch_pauli_reduce(r, nrows, s), "Pauli reduce launch");
    }
}

// Run the Pauli kernel over group gi's rows: expectations into out[b, k]
// (when out is not NULL) and, when phi is not NULL, phi = sum_k g_k h_k psi
// with g = upstream.  Observables are split over launches so that the
// per-workgroup partials stay within a bounded workspace.
// phi = g H psi and <psi|H|psi> of a single observable (K = 1) with the
// kernels generated for it: one read of psi and one update of phi per pass.
// phi = g H psi and <psi|H|psi> of a single observable (K = 1) with the
// kernels generated for it.
void spec_phi_group(tq_program p, size_t gi, const float2 *psi, float2 *phi, const float *upstream, float *out,
                    hipStream_t s)
{
    const Group &g = *p->pd->groups[gi];
    GroupDev &gd = *p->gdev[gi];
    ObsGroupDev &og = *p->obs_dev[gi];
    const int nrows = (int)g.rows.size();
    const int npass = (int)og.phi_passes.size();
    HPhiArgs a{};
    a.psi = psi;
    a.phi = phi;
    a.row_stride = (int64_t)1 << g.n;
    a.rows = (const int32_t *)gd.ident.p;
    a.brows = (const int32_t *)gd.rows.p;
    a.upstream = upstream;
    a.K = 1;
    a.wg_per_row = wg_for(nrows, g.n - og.phi_passes[0].geom.t);
    a.npass = npass;
    a.partial = (double *)p->partial.ensure(sizeof(double) * (size_t)nrows * npass * a.wg_per_row);
    std::string log;
    for (int pi = 0; pi < npass; pi++) {
        a.g = og.phi_passes[pi].geom;
        a.pass = pi;
        const hipError_t e = launch_hphi_spec(og.phi_src, pi, a, nrows, s, &log, &og.phi_memo);
        if (e == hipErrorInvalidSource) fail(TQ_E_DEVICE, log);
        hip_check(e, "specialised H_g launch");
    }
    if (!out) return;
    PauliReduceArgs r{};
    r.rows = (const int32_t *)gd.rows.p;
    r.partial = a.partial;
    r.wg_per_row = npass * a.wg_per_row;  // the passes' workgroups side by side
    r.K = 1;
    r.k_begin = 0;
    r.k_count = 1;
    r.out = out;
    hip_check(launch_pauli_reduce(r, nrows, s), "Pauli reduce launch");
}

void pauli_group(tq_program p, size_t gi, const float2 *psi, float2 *phi, const float *upstream, int K, float *out,
                 hipStream_t s, const RunRows &rr)
{
    const Group &g = *p->pd->groups[gi];
    ObsGroupDev &og = *p->obs_dev[gi];
    const int nrows = rr.n;
    if (K == 0 || nrows == 0) return;
    if (!phi && og.diag) {
        diag_group(p, gi, psi, K, out, s, rr);
        return;
    }
    if (!phi && !og.spec_sets.empty()) {
        spec_pauli_group(p, gi, psi, K, out, s, rr);
        return;
    }
    if (phi && upstream && K == 1 && !og.phi_passes.empty() && rr.period == 0) {
        spec_phi_group(p, gi, psi, phi, upstream, out, s);
        return;
    }
    PauliArgs a{};
    a.psi = psi;
    a.phi = phi;
    a.row_stride = (int64_t)1 << g.n;
    a.rows = rr.ident;
    a.brows = rr.out_rows;
    a.chunks = (const PChunk *)og.chunks.p;
    a.row_chunk_begin = or_own<int32_t>(rr.cbegin, og.cbegin);
    a.row_chunk_count = or_own<int32_t>(rr.ccount, og.ccount);
    a.xfg = (const PXfGroup *)og.xfg.p;
    a.xg = (const PXGroup *)og.xg.p;
    a.us = (const PUSub *)og.us.p;
    a.terms = (const PTerm *)og.pterms.p;
    a.upstream = upstream;
    a.K = K;
    a.g = og.pgeom;
    a.tiles_log2 = g.n - og.pgeom.t;
    // every tile of a row in flight at once (partner tiles then come from L2),
    // up to 2^18 workgroups per launch
    const int64_t ntiles = (int64_t)1 << a.tiles_log2;
    a.wg_per_row = (int)std::max<int64_t>(1, std::min<int64_t>(ntiles, ((int64_t)1 << 18) / nrows));
    const int64_t slots = (int64_t)nrows * a.wg_per_row;
    const int kmax = (int)std::max<int64_t>(
        kPauliChunk, std::min<int64_t>(1024, ((int64_t)32 << 20) / slots) / kPauliChunk * kPauliChunk);
    for (int k0 = 0; k0 < K; k0 += kmax) {
        a.k_begin = k0;
        a.k_count = std::min(kmax, K - k0);
        a.phi_accumulate = k0 > 0;
        a.partial = (double *)p->partial.ensure(sizeof(double) * (size_t)slots * a.k_count);
        hip_check(launch_pauli(a, nrows, og.partner, s), "Pauli kernel launch");
        if (out) {
            PauliReduceArgs r{};
            r.rows = a.brows;
            r.partial = a.partial;
            r.wg_per_row = a.wg_per_row;
            r.K = K;
            r.k_begin = k0;
            r.k_count = a.k_count;
            r.out = out;
            hip_check(launch_pauli_reduce(r, nrows, s), "Pauli reduce launch");
        }
    }
}

hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

// Small circuits run as one resident kernel per call when psi (and phi), the
// row's matrices and the accumulators fit in LDS.
constexpr size_t kResidentLds = 150 * 1024;
// the specialised resident kernel is launched with at most the default
// dynamic LDS window
constexpr size_t kResidentSpecLds = 64 * 1024;

bool resident(tq_program p, size_t gi, bool adjoint, int tmax)
{
    const Group &g = *p->pd->groups[gi];
    if (g.n > std::min(p->pd->opt.tile, 12)) return false;
    const int nacc = std::max(tmax + (adjoint ? g.n_gslots : 0), 1);
    const size_t lds = resident_lds_bytes(g.n, nacc, adjoint);
    // the precompiled resident kernel runs reverse stages of at most
    // kStageBitsRevResident bits; wider ones need the specialised kernel
    for (const Pass &ps : g.rev)
        for (const Stage &st : ps.stages)
            if (st.r > kStageBitsRevResident && !(p->pd->opt.specialize && lds <= kResidentSpecLds)) return false;
    return lds <= kResidentLds;
}

// Launch the resident kernel of group gi: the one specialised for the
// group's structure when the program asks for it and its LDS fits the
// default window, else the precompiled one.
void run_resident(tq_program p, size_t gi, const ResArgs &a, int nrows, hipStream_t s)
{
    const Group &g = *p->pd->groups[gi];
    const size_t lds = resident_lds_bytes(a.n, a.nacc, a.grad != nullptr);
    if (p->pd->opt.specialize && lds <= kResidentSpecLds) {
        std::string log;
        const hipError_t e = launch_resident_spec(g, a, nrows, lds, s, &log, &p->gdev[gi]->res_memo);
        if (e == hipErrorInvalidSource) fail(TQ_E_DEVICE, log);
        hip_check(e, "specialised resident launch");
        return;
    }
    hip_check(launch_resident(a, nrows, s), "resident launch");
}

ResArgs resident_args(tq_program p, size_t gi, const float *theta, bool adjoint, hipStream_t s, const RunRows &rr)
{
    const Group &g = *p->pd->groups[gi];
    GroupDev &gd = *p->gdev[gi];
    build_mats(p, gi, theta, g.fwd_tasks.begin, adjoint ? g.rev_tasks.end : g.fwd_tasks.end, s, rr);
    ResArgs a{};
    a.mats = rr.mats;
    a.mat_stride = std::max(g.mat_block, 1);
    a.slot_scale = (const double *)gd.scale.p;
    a.uniform = g.uniform_slots;
    a.n_slots = g.n_slots;
    a.S = p->pd->S;
    a.rows = rr.out_rows;
    a.n = g.n;
    a.fops = (const PassOp *)gd.fwd_ops.p;
    a.fstages = (const Stage *)gd.fwd_stages.p;
    a.nfstages = gd.n_fwd_stages;
    for (int q = 0; q < kMaxQubits; q++) a.init_mat[q] = g.init_mat[q];
    a.rops = (const PassOp *)gd.rev_ops.p;
    a.rstages = (const Stage *)gd.rev_stages.p;
    a.nrstages = gd.n_rev_stages;
    a.sym_begin = (const int32_t *)gd.sym_begin.p;
    a.sym_gslots = (const int32_t *)gd.sym_gslots.p;
    a.gslot_slot = (const int32_t *)gd.gslot_slot.p;
    a.nacc = 1;
    return a;
}

void resident_terms(tq_program p, size_t gi, ResArgs &a, int K, float *exp_out, const RunRows &rr)
{
    ObsGroupDev &og = *p->obs_dev[gi];
    a.terms = (const TermDev *)og.terms.p;
    a.row_term_begin = or_own<int32_t>(rr.term_begin, og.begin);
    a.row_term_count = or_own<int32_t>(rr.term_count, og.count);
    a.K = K;
    a.exp_out = exp_out;
    a.gacc = og.tmax;
    a.nacc = std::max(og.tmax, 1);
}

// the final states of group gi into its rows of the state workspace
void forward_to_ws(tq_program p, size_t gi, const float *theta, float2 *psi, hipStream_t s, const RunRows &rr)
{
    const Group &g = *p->pd->groups[gi];
    if (resident(p, gi, false, 0)) {
        ResArgs a = resident_args(p, gi, theta, false, s, rr);
        a.state_out = psi;
        a.out_stride = (int64_t)1 << g.n;
        a.out_rows = rr.ident;
        run_resident(p, gi, a, rr.n, s);
        return;
    }
    build_mats(p, gi, theta, g.fwd_tasks.begin, g.fwd_tasks.end, s, rr);
    forward(p, gi, psi, (int64_t)1 << g.n, rr.ident, s, rr);
}


void check_align(const void *p, size_t a, const char *name)
{
    if (reinterpret_cast<uintptr_t>(p) % a != 0)
        fail(TQ_E_INVALID, std::string(name) + " must be " + std::to_string(a) + "-byte aligned");
}

void fill_levels(SampArgs &a, int n)
{
    a.count[0] = (int64_t)1 << n;
    a.off[0] = 0;
    int k = 0;
    int64_t total = 0;
    while (a.count[k] > 64) {
        a.count[k + 1] = (a.count[k] + 63) / 64;
        a.off[k + 1] = total;
        total += a.count[k + 1];
        k++;
    }
    a.nlev = k;
    a.row_level = std::max<int64_t>(total, 1);
}

// ---------------------------------------------- sampled expectations
// Limits of the shot counter ((e K + k) 2^40 + t 2^24 + s): e K + k < 2^24,
// t < 2^16, s < 2^24.
constexpr int64_t kMaxCounterRows = (int64_t)1 << 24;

// The term observables and shot tables of an observables handle, built on
// first use (tables on the current device).
void prepare_terms(tq_observables o)
{
    int dev = -1;
    hip_check(hipGetDevice(&dev), "hipGetDevice");
    if (o->terms) {
        if (dev != o->dev) fail(TQ_E_INVALID, "observables were first used on another device");
        return;
    }
    const ObsData &od = *o->od;
    auto t = std::make_unique<ObsData>();
    t->B = od.B;
    int Kt = 0;
    for (int b = 0; b < od.B; b++) {
        int n = 0;
        for (int k = 0; k < od.K; k++) {
            const auto &sum = od.sums[(size_t)b * od.K + k];
            if (sum.size() >= ((size_t)1 << 16)) fail(TQ_E_UNSUPPORTED, "sampled expectation: more than 65535 terms in one observable");
            for (const HTerm &h : sum) n += !h.factors.empty();
        }
        Kt = std::max(Kt, n);
    }
    t->K = Kt;
    t->sums.resize((size_t)od.B * Kt);
    // tables: per row the (k, t) of each slot and per observable its terms
    bool uniform = true;
    for (int b = 1; b < od.B && uniform; b++)
        for (int k = 0; k < od.K && uniform; k++) {
            const auto &x = od.sums[k], &y = od.sums[(size_t)b * od.K + k];
            uniform = x.size() == y.size();
            for (size_t i = 0; i < x.size() && uniform; i++)
                uniform = x[i].coeff == y[i].coeff && x[i].factors == y[i].factors;
        }
    const int tb = uniform ? std::min(od.B, 1) : od.B;  // table rows
    size_t tmax = 0;
    for (int b = 0; b < tb; b++) {
        size_t n = 0;
        for (int k = 0; k < od.K; k++) n += od.sums[(size_t)b * od.K + k].size();
        tmax = std::max(tmax, n);
    }
    std::vector<int32_t> slot_k((size_t)tb * Kt, 0), slot_t((size_t)tb * Kt, -1), obs_begin((size_t)tb * (od.K + 1));
    std::vector<int32_t> term_slot(std::max<size_t>((size_t)tb * tmax, 1), -1);
    std::vector<double> term_coeff(term_slot.size(), 0.0);
    for (int b = 0; b < od.B; b++) {
        int j = 0;
        size_t ti = 0;
        for (int k = 0; k < od.K; k++) {
            const auto &sum = od.sums[(size_t)b * od.K + k];
            if (b < tb) obs_begin[(size_t)b * (od.K + 1) + k] = (int32_t)ti;
            for (size_t tt = 0; tt < sum.size(); tt++, ti++) {
                const HTerm &h = sum[tt];
                if (b < tb) term_coeff[(size_t)b * tmax + ti] = h.coeff;
                if (h.factors.empty()) continue;
                t->sums[(size_t)b * Kt + j].push_back(HTerm{1.0, h.factors});
                if (b < tb) {
                    slot_k[(size_t)b * Kt + j] = k;
                    slot_t[(size_t)b * Kt + j] = (int32_t)tt;
                    term_slot[(size_t)b * tmax + ti] = j;
                }
                j++;
            }
        }
        if (b < tb) obs_begin[(size_t)b * (od.K + 1) + od.K] = (int32_t)ti;
    }
    t->id = g_obs_counter.fetch_add(1);
    upload(o->slot_k, slot_k);
    upload(o->slot_t, slot_t);
    upload(o->obs_begin, obs_begin);
    upload(o->term_slot, term_slot);
    upload(o->term_coeff, term_coeff);
    o->term_stride = (int64_t)tmax;
    o->uniform = uniform;
    o->Kt = Kt;
    o->dev = dev;
    o->terms = std::move(t);
}

SampledArgs sampled_args(tq_observables o, int reps, uint64_t seed)
{
    SampledArgs a{};
    a.Kt = o->Kt;
    a.K = o->od->K;
    a.reps = reps;
    a.seed = seed;
    a.slot_k = (const int32_t *)o->slot_k.p;
    a.slot_t = (const int32_t *)o->slot_t.p;
    a.slot_stride = o->uniform ? 0 : o->Kt;
    a.obs_begin = (const int32_t *)o->obs_begin.p;
    a.obs_stride = o->uniform ? 0 : o->od->K + 1;
    a.term_slot = (const int32_t *)o->term_slot.p;
    a.term_coeff = (const double *)o->term_coeff.p;
    a.term_stride = o->uniform ? 0 : o->term_stride;
    return a;
}

// Expectations of every group's rows (the body of tq_expectation).
void expectations_all(tq_program prog, const float *theta, const ObsData &od, float *out, hipStream_t s)
{
    const ProgramData &pd = *prog->pd;
    ensure_obs(prog, od);
    float2 *psi = psi_ws(prog);
    for (size_t gi = 0; gi < pd.groups.size(); gi++) {
        const Group &g = *pd.groups[gi];
        GroupDev &gd = *prog->gdev[gi];
        const RunRows rr = own_rows(prog, gi);
        if (resident(prog, gi, false, prog->obs_dev[gi]->tmax)) {
            ResArgs a = resident_args(prog, gi, theta, false, s, rr);
            resident_terms(prog, gi, a, od.K, out, rr);
            run_resident(prog, gi, a, rr.n, s);
            continue;
        }
        build_mats(prog, gi, theta, g.fwd_tasks.begin, g.fwd_tasks.end, s, rr);
        forward(prog, gi, psi + gd.psi_off, (int64_t)1 << g.n, rr.ident, s, rr);
        pauli_group(prog, gi, psi + gd.psi_off, nullptr, nullptr, od.K, out, s, rr);
    }
}

// ------------------------------------------------ batched shift rules
enum ShiftKind { kParamShift = 0, kFiniteDiff = 1 };
// derived rows copy their source row's matrices (and rebuild only the moved
// tasks) when the expansion would otherwise build at least this many tasks
constexpr int64_t kDerivedCopyTasks = (int64_t)1 << 20;

// The derived rows of group gi for one kind: parameter shift, pair p = the
// p-th symbolic blob parameter moved by +delta (row 2p) and -delta (row
// 2p + 1), gradient coefficient factor / mult x the row's scale of its
// first slot; central differences, pair p = the p-th symbol the group uses
// moved by +-eps (the moves are +-1 times eps), coefficient 1 / (2 eps)
// applied at the reduction.
void ensure_x(tq_program p, size_t gi, int kind)
{
    GroupDev &gd = *p->gdev[gi];
    if (gd.x_ready[kind]) return;
    const Group &g = *p->pd->groups[gi];
    const int S = p->pd->S;
    std::vector<ShiftDev> sh;
    std::vector<int32_t> pslot, psym;
    std::vector<double> pcoef;
    if (kind == kParamShift) {
        for (const Occurrence &oc : g.occurrences) {
            double delta, factor;
            if (!shift_rule(oc.blob_op, oc.param, &delta, &factor))
                fail(TQ_E_UNSUPPORTED, "parameter shift: a symbolic parameter has no two-term shift rule "
                                       "(fSim theta; use the adjoint or finite differences)");
            for (int sg : {1, -1}) {
                ShiftDev d{};
                d.slot[0] = oc.slot[0];
                d.slot[1] = oc.slot[1];
                d.sym = -1;
                d.delta[0] = sg * oc.mult[0] * delta;
                d.delta[1] = oc.slot[1] >= 0 ? sg * oc.mult[1] * delta : 0.0;
                sh.push_back(d);
            }
            pslot.push_back(oc.slot[0]);
            pcoef.push_back(factor / oc.mult[0]);
            psym.push_back(oc.sym);
        }
    } else {
        std::vector<char> used(S, 0);
        for (int32_t sy : g.slot_sym)
            if (sy >= 0) used[sy] = 1;
        for (int sy = 0; sy < S; sy++) {
            if (!used[sy]) continue;
            for (int sg : {1, -1}) {
                ShiftDev d{};
                d.slot[0] = d.slot[1] = -1;
                d.sym = sy;
                d.dtheta = sg;
                sh.push_back(d);
            }
            pslot.push_back(-1);
            pcoef.push_back(1.0);
            psym.push_back(sy);
        }
    }
    // per move the forward build tasks that read a moved parameter (any
    // member gate with a moved slot, or a slot of the moved symbol).  When
    // the row carries a global phase: if the first qubit's product-init task
    // is among them it heads the list and takes the moved row's whole phase;
    // else its copied matrix keeps the source row's phase times the change
    // of the phase terms of the moved parameters (listed per move)
    auto slot_moved = [&](const ShiftDev &d, int sl) {
        return sl >= 0 && (sl == d.slot[0] || sl == d.slot[1] || (d.sym >= 0 && g.slot_sym[sl] == d.sym));
    };
    auto task_moved = [&](const ShiftDev &d, int ti) {
        const BuildTask &bt = g.tasks[ti];
        for (int mi = 0; mi < bt.mem_count; mi++) {
            const GateDev &gd0 = g.gates[g.members[bt.mem_begin + mi].gate];
            for (int j = 0; j < gd0.np; j++)
                if (slot_moved(d, gd0.slot0 + j)) return true;
        }
        return false;
    };
    std::vector<int32_t> lbegin(1, 0), list, pfull, pbegin(1, 0), plist;
    int init_task = -1;
    for (int ti = g.fwd_tasks.begin; ti < g.fwd_tasks.end; ti++)
        if (g.n > 0 && g.tasks[ti].out == g.init_mat[0]) init_task = ti;
    int max_list = 0;
    for (const ShiftDev &d : sh) {
        const size_t at = list.size();
        const bool full = !g.phase_terms.empty() && init_task >= 0 && task_moved(d, init_task);
        if (full) list.push_back(init_task);
        for (int ti = g.fwd_tasks.begin; ti < g.fwd_tasks.end; ti++)
            if (!(full && ti == init_task) && task_moved(d, ti)) list.push_back(ti);
        max_list = std::max(max_list, (int)(list.size() - at));
        lbegin.push_back((int32_t)list.size());
        pfull.push_back(full ? 1 : 0);
        if (!full)
            for (size_t j = 0; j < g.phase_terms.size(); j++)
                if (slot_moved(d, g.phase_terms[j].slot)) plist.push_back((int32_t)j);
        pbegin.push_back((int32_t)plist.size());
    }
    upload(gd.x_list_begin[kind], lbegin);
    upload(gd.x_list[kind], list);
    upload(gd.x_phase_full[kind], pfull);
    upload(gd.x_phase_begin[kind], pbegin);
    upload(gd.x_phase_list[kind], plist);
    gd.x_max_list[kind] = max_list;
    std::vector<int32_t> begin(S + 1, 0), pairs(psym.size());
    for (int32_t sy : psym) begin[sy + 1]++;
    for (int i = 0; i < S; i++) begin[i + 1] += begin[i];
    std::vector<int32_t> fill(begin.begin(), begin.end() - 1);
    for (size_t pi = 0; pi < psym.size(); pi++) pairs[fill[psym[pi]]++] = (int32_t)pi;
    upload(gd.x_shift[kind], sh);
    upload(gd.x_pair_slot[kind], pslot);
    upload(gd.x_pair_coef[kind], pcoef);
    upload(gd.x_sym_begin[kind], begin);
    upload(gd.x_sym_pairs[kind], pairs);
    gd.x_period[kind] = (int)sh.size();
    gd.x_ready[kind] = true;
}

// Shot-counter rows of the parameter-shift rows: the shifted circuits of all
// rows as one batch in row order, each row's 2 x (its occurrences) in
// (occurrence, +/-) order; per group row the first of its row.
int64_t ensure_ebase(tq_program p)
{
    const ProgramData &pd = *p->pd;
    std::vector<int64_t> per_row(pd.B, 0);
    for (size_t gi = 0; gi < pd.groups.size(); gi++)
        for (int32_t b : pd.groups[gi]->rows) per_row[b] = 2 * (int64_t)pd.groups[gi]->occurrences.size();
    std::vector<int64_t> start(pd.B + 1, 0);
    for (int b = 0; b < pd.B; b++) start[b + 1] = start[b] + per_row[b];
    for (size_t gi = 0; gi < pd.groups.size(); gi++) {
        GroupDev &gd = *p->gdev[gi];
        if (gd.x_ebase.p) continue;
        std::vector<int64_t> e;
        for (int32_t b : pd.groups[gi]->rows) e.push_back(start[b]);
        upload(gd.x_ebase, e);
    }
    return start[pd.B];
}

const int32_t *ident_rows(tq_program p, int n)
{
    if (p->xident_n < n) {
        std::vector<int32_t> v(n);
        for (int i = 0; i < n; i++) v[i] = i;
        upload(p->xident, v);
        p->xident_n = n;
    }
    return (const int32_t *)p->xident.p;
}

// Derived rows per launch: at most 65535 (one grid row each in the builder),
// states within 4 GiB and matrices within 1 GiB.
int derived_chunk(tq_program p, size_t gi, int64_t total, bool on_chip)
{
    const Group &g = *p->pd->groups[gi];
    int64_t c = std::min<int64_t>(total, 65535);
    c = std::min<int64_t>(c, std::max<int64_t>(1, ((int64_t)1 << 30) / (16 * (int64_t)std::max(g.mat_block, 1))));
    if (!on_chip) c = std::min<int64_t>(c, std::max<int64_t>(1, ((int64_t)1 << 32) / ((int64_t)8 << g.n)));
    return (int)std::max<int64_t>(c, 1);
}

// Gradients of sum_k g_k <h_k> of every row by a batched shift rule: the
// derived rows of each group run chunk by chunk through the same build,
// forward and expectation kernels as plain rows (reps > 0: their sampled
// expectations), then one reduction per group forms the gradients.
void shift_grad(tq_program prog, const float *theta, tq_observables obs, const float *upstream, int kind, int reps,
                uint64_t seed, double eps, float *grad, hipStream_t s)
{
    const ProgramData &pd = *prog->pd;
    const ObsData &od = *obs->od;
    const int K = od.K;
    for (size_t gi = 0; gi < pd.groups.size(); gi++) ensure_x(prog, gi, kind);
    if (reps > 0) {
        prepare_terms(obs);
        const int64_t total = ensure_ebase(prog);
        if (total * (int64_t)std::max(K, 1) >= kMaxCounterRows)
            fail(TQ_E_UNSUPPORTED, "sampled parameter shift: too many (shifted circuit, observable) pairs for the "
                                   "shot counter (2^24)");
    }
    const ObsData &eod = reps > 0 ? *obs->terms : od;  // observables the derived rows evaluate
    const int Ke = eod.K;
    ensure_obs(prog, eod);
    // workspaces sized for the largest group first (none is reallocated
    // while work of an earlier group may still read it)
    size_t need_out = 1, need_mats = 1, need_psi = 1, need_chunk = 1;
    std::vector<int> chunks(pd.groups.size(), 0);
    std::vector<char> on_chip(pd.groups.size(), 0);
    for (size_t gi = 0; gi < pd.groups.size(); gi++) {
        const Group &g = *pd.groups[gi];
        const int64_t total = (int64_t)g.rows.size() * prog->gdev[gi]->x_period[kind];
        if (total == 0 || K == 0) continue;
        on_chip[gi] = resident(prog, gi, false, prog->obs_dev[gi]->tmax);
        chunks[gi] = derived_chunk(prog, gi, total, on_chip[gi]);
        need_out = std::max(need_out, (size_t)total * K);
        need_mats = std::max(need_mats, (size_t)chunks[gi] * std::max(g.mat_block, 1));
        if (!on_chip[gi]) need_psi = std::max(need_psi, (size_t)chunks[gi] << g.n);
        need_chunk = std::max(need_chunk, (size_t)chunks[gi]);
    }
    float *f_all = (float *)prog->xout.ensure(sizeof(float) * need_out);
    double2 *mats = (double2 *)prog->xmats.ensure(sizeof(double2) * need_mats);
    float2 *psi = need_psi > 1 ? (float2 *)prog->xpsi.ensure(sizeof(float2) * need_psi) : nullptr;
    const int32_t *ident = ident_rows(prog, (int)need_chunk);
    float *tv = reps > 0 ? (float *)prog->xterm.ensure(sizeof(float) * need_chunk * std::max(Ke, 1)) : nullptr;
    uint32_t *counts = reps > 0 ? (uint32_t *)prog->xcounts.ensure(sizeof(uint32_t) * need_chunk * std::max(Ke, 1))
                                : nullptr;
    int32_t *tab_buf[kRowGatherArrays];
    for (int j = 0; j < kRowGatherArrays; j++) tab_buf[j] = (int32_t *)prog->xtab[j].ensure(sizeof(int32_t) * need_chunk);
    for (size_t gi = 0; gi < pd.groups.size(); gi++) {
        const Group &g = *pd.groups[gi];
        GroupDev &gd = *prog->gdev[gi];
        ObsGroupDev &og = *prog->obs_dev[gi];
        const int nrows = (int)g.rows.size();
        const int period = gd.x_period[kind];
        const int64_t total = (int64_t)nrows * period;
        float *f = nullptr;
        if (total > 0 && K > 0) {
            f = f_all;
            const int chunk = chunks[gi];
            // large expansions: the source rows' forward matrices, which
            // every derived row copies before its moved tasks are built again
            // (small ones build every task, in fewer launches)
            const bool copy_build =
                (int64_t)total * (g.fwd_tasks.end - g.fwd_tasks.begin) >= kDerivedCopyTasks;
            if (copy_build) build_mats(prog, gi, theta, g.fwd_tasks.begin, g.fwd_tasks.end, s, own_rows(prog, gi));
            // per-row observable tables, gathered from the source rows
            const DevBuf *tab_in[kRowGatherArrays] = {&og.begin, &og.count, &og.cbegin, &og.ccount, &og.dcbegin,
                                                      &og.dccount};
            int32_t *tab_out[kRowGatherArrays];
            for (int j = 0; j < kRowGatherArrays; j++) tab_out[j] = tab_in[j]->p ? tab_buf[j] : nullptr;
            for (int64_t begin = 0; begin < total; begin += chunk) {
                const int c = (int)std::min<int64_t>(chunk, total - begin);
                RunRows rr;
                rr.n = c;
                rr.begin = begin;
                rr.period = period;
                rr.shift = (const ShiftDev *)gd.x_shift[kind].p;
                rr.eps = eps;
                if (copy_build) {
                    rr.x_src = mat_ws(prog) + gd.mat_off;
                    rr.list_begin = (const int32_t *)gd.x_list_begin[kind].p;
                    rr.task_list = (const int32_t *)gd.x_list[kind].p;
                    rr.phase_full = (const int32_t *)gd.x_phase_full[kind].p;
                    rr.phase_begin = (const int32_t *)gd.x_phase_begin[kind].p;
                    rr.phase_list = (const int32_t *)gd.x_phase_list[kind].p;
                    rr.max_list = gd.x_max_list[kind];
                }
                rr.mats = mats;
                rr.ident = ident;
                rr.out_rows = ident;
                RowGatherArgs ra{};
                for (int j = 0; j < kRowGatherArrays; j++)
                    if (tab_out[j]) {
                        ra.in[ra.narrays] = (const int32_t *)tab_in[j]->p;
                        ra.out[ra.narrays] = tab_out[j];
                        ra.narrays++;
                    }
                ra.x_begin = begin;
                ra.x_period = period;
                ra.count = c;
                hip_check(launch_row_gather(ra, s), "row table gather launch");
                rr.term_begin = tab_out[0];
                rr.term_count = tab_out[1];
                rr.cbegin = tab_out[2];
                rr.ccount = tab_out[3];
                rr.dcbegin = tab_out[4];
                rr.dccount = tab_out[5];
                float *vals = reps > 0 ? tv : f + begin * K;
                if (Ke > 0) {
                    if (on_chip[gi]) {
                        ResArgs a = resident_args(prog, gi, theta, false, s, rr);
                        resident_terms(prog, gi, a, Ke, vals, rr);
                        run_resident(prog, gi, a, c, s);
                    } else {
                        build_mats(prog, gi, theta, g.fwd_tasks.begin, g.fwd_tasks.end, s, rr);
                        forward(prog, gi, psi, (int64_t)1 << g.n, ident, s, rr);
                        pauli_group(prog, gi, psi, nullptr, nullptr, Ke, vals, s, rr);
                    }
                }
                if (reps > 0) {
                    SampledArgs sa = sampled_args(obs, reps, seed);
                    sa.tv = tv;
                    sa.rows = (const int32_t *)gd.rows.p;
                    sa.ebase = (const int64_t *)gd.x_ebase.p;
                    sa.x_begin = begin;
                    sa.x_period = period;
                    sa.nrows = c;
                    sa.counts = counts;
                    sa.out = f + begin * K;
                    hip_check(launch_sampled(sa, s), "sampled expectation launch");
                }
            }
        }
        ShiftGradArgs ga{};
        ga.f = f;
        ga.K = K;
        ga.S = pd.S;
        ga.period = period;
        ga.rows = (const int32_t *)gd.rows.p;
        ga.upstream = upstream;
        ga.sym_begin = (const int32_t *)gd.x_sym_begin[kind].p;
        ga.sym_pairs = (const int32_t *)gd.x_sym_pairs[kind].p;
        ga.pair_slot = (const int32_t *)gd.x_pair_slot[kind].p;
        ga.pair_coef = (const double *)gd.x_pair_coef[kind].p;
        ga.coef_mul = kind == kFiniteDiff ? 1.0 / (2.0 * eps) : 1.0;
        ga.slot_scale = (const double *)gd.scale.p;
        ga.uniform = g.uniform_slots;
        ga.n_slots = g.n_slots;
        ga.grad = grad;
        hip_check(launch_shift_grad(ga, nrows, s), "shift-rule gradient launch");
    }
}

} // namespace

// ------------------------------------------------------------------- ABI
extern "C" {

const char *tq_last_error(void) { return g_err.c_str(); }
const char *tq_version(void) { return "tq 0.1 (gfx950)"; }

tq_status tq_program_create(const void *blob, size_t nbytes, const tq_options *opt, tq_program *out)
{
    return guarded([&] {
        if (!out) fail(TQ_E_INVALID, "out is NULL");
        *out = nullptr;
        Options o;
        if (opt) {
            if (opt->max_tile_qubits) {
                if (opt->max_tile_qubits < 8 || opt->max_tile_qubits > 13)
                    fail(TQ_E_INVALID, "max_tile_qubits must be in 8..13");
                o.tile = opt->max_tile_qubits;
            }
            if (opt->low_qubits) {
                if (opt->low_qubits < 3 || opt->low_qubits > 8) fail(TQ_E_INVALID, "low_qubits must be in 3..8");
                o.low = opt->low_qubits;
            }
            if (opt->fuse < 0) o.fuse = false;
            if (opt->max_pass_gates < 0) fail(TQ_E_INVALID, "max_pass_gates must be >= 0");
            o.max_pass_gates = opt->max_pass_gates;
            if (opt->specialize < 0 || opt->specialize > 1) fail(TQ_E_INVALID, "specialize must be 0 or 1");
            o.specialize = opt->specialize == 1;
        }
        // generated passes default to tiles of 2^13 amplitudes: fewer passes
        // for the same gates (measured: the 30-qubit random circuit 46 -> 40
        // passes, 181 -> 163 ms; QAOA 9.9 -> 8.7 ms; VQE 85 -> 83 ms)
        if (o.specialize && !(opt && opt->max_tile_qubits)) o.tile = 13;
        if (o.low > o.tile - 2) o.low = o.tile - 2;
        auto p = std::make_unique<tq_program_s>();
        p->pd = parse_program(blob, nbytes, o);
        *out = p.release();
    });
}

void tq_program_destroy(tq_program prog) { delete prog; }

tq_status tq_program_info(tq_program prog, int32_t *B, int32_t *S, int32_t *max_qubits, int32_t *qpc)
{
    return guarded([&] {
        if (!prog) fail(TQ_E_INVALID, "program is NULL");
        if (B) *B = prog->pd->B;
        if (S) *S = prog->pd->S;
        if (max_qubits) *max_qubits = prog->pd->nmax;
        if (qpc)
            for (int b = 0; b < prog->pd->B; b++) qpc[b] = prog->pd->circuits[b].n;
    });
}

tq_status tq_program_set_noise_seed(tq_program prog, uint64_t seed)
{
    return guarded([&] {
        if (!prog) fail(TQ_E_INVALID, "program is NULL");
        prog->noise_seed = seed;
    });
}

tq_status tq_row_mean(const float *in, int64_t groups, int32_t R, int32_t K, float *out, void *stream)
{
    return guarded([&] {
        if (groups < 0 || R < 1 || K < 0) fail(TQ_E_INVALID, "row_mean: groups >= 0, R >= 1 and K >= 0 required");
        if (groups == 0 || K == 0) return;
        if (!in || !out) fail(TQ_E_INVALID, "row_mean: in and out must not be NULL");
        check_align(in, 4, "in");
        check_align(out, 4, "out");
        hip_check(launch_row_mean(in, groups, R, K, out, as_stream(stream)), "row mean launch");
    });
}

tq_status tq_program_specialize(tq_program prog, const char *target)
{
    return guarded([&] {
        if (!prog) fail(TQ_E_INVALID, "program is NULL");
        if (!prog->pd->opt.specialize) return;
        for (size_t gi = 0; gi < prog->pd->groups.size(); gi++) {
            std::string log;
            const hipError_t e = prepare_spec(*prog->pd->groups[gi], resident(prog, gi, false, 0), target, &log);
            if (e == hipErrorInvalidSource) fail(TQ_E_DEVICE, log);
            hip_check(e, "specialised kernel compilation");
        }
    });
}

tq_status tq_observables_create(const void *blob, size_t nbytes, tq_observables *out)
{
    return guarded([&] {
        if (!out) fail(TQ_E_INVALID, "out is NULL");
        *out = nullptr;
        auto o = std::make_unique<tq_observables_s>();
        o->od = parse_observables(blob, nbytes);
        o->od->id = g_obs_counter.fetch_add(1);
        *out = o.release();
    });
}

void tq_observables_destroy(tq_observables obs) { delete obs; }

tq_status tq_observables_info(tq_observables obs, int32_t *B, int32_t *K)
{
    return guarded([&] {
        if (!obs) fail(TQ_E_INVALID, "observables handle is NULL");
        if (B) *B = obs->od->B;
        if (K) *K = obs->od->K;
    });
}

tq_status tq_simulate_state(tq_program prog, const float *theta, void *states, void *stream)
{
    return guarded([&] {
        if (!prog) fail(TQ_E_INVALID, "program is NULL");
        const ProgramData &pd = *prog->pd;
        if (pd.B == 0) return;
        if (!states) fail(TQ_E_INVALID, "states is NULL");
        if (pd.S > 0 && !theta) fail(TQ_E_INVALID, "symbol_values is NULL");
        check_align(states, 16, "states");
        check_align(theta, 4, "symbol_values");
        ensure_device(prog);
        hipStream_t s = as_stream(stream);
        const int64_t stride = (int64_t)1 << pd.nmax;
        for (size_t gi = 0; gi < pd.groups.size(); gi++) {
            const Group &g = *pd.groups[gi];
            GroupDev &gd = *prog->gdev[gi];
            const RunRows rr = own_rows(prog, gi);
            if (resident(prog, gi, false, 0)) {
                ResArgs a = resident_args(prog, gi, theta, false, s, rr);
                a.state_out = (float2 *)states;
                a.out_stride = stride;
                a.out_rows = (const int32_t *)gd.rows.p;
                run_resident(prog, gi, a, rr.n, s);
            } else {
                build_mats(prog, gi, theta, g.fwd_tasks.begin, g.fwd_tasks.end, s, rr);
                forward(prog, gi, (float2 *)states, stride, (const int32_t *)gd.rows.p, s, rr);
            }
            if (g.n < pd.nmax)
                hip_check(launch_zero_tail((float2 *)states, stride, (const int32_t *)gd.rows.p, (int)g.rows.size(),
                                           (int64_t)1 << g.n, stride, s),
                          "zero tail launch");
        }
    });
}

tq_status tq_expectation(tq_program prog, const float *theta, tq_observables obs, float *out, void *stream)
{
    return guarded([&] {
        if (!prog || !obs) fail(TQ_E_INVALID, "program or observables is NULL");
        const ProgramData &pd = *prog->pd;
        check_obs_fit(prog, obs);
        if (pd.B == 0 || obs->od->K == 0) return;
        if (!out) fail(TQ_E_INVALID, "out is NULL");
        if (pd.S > 0 && !theta) fail(TQ_E_INVALID, "symbol_values is NULL");
        check_align(out, 4, "out");
        check_align(theta, 4, "symbol_values");
        ensure_device(prog);
        ensure_obs(prog, *obs->od);
        hipStream_t s = as_stream(stream);
        float2 *psi = psi_ws(prog);
        for (size_t gi = 0; gi < pd.groups.size(); gi++) {
            const Group &g = *pd.groups[gi];
            GroupDev &gd = *prog->gdev[gi];
            const RunRows rr = own_rows(prog, gi);
            if (resident(prog, gi, false, prog->obs_dev[gi]->tmax)) {
                ResArgs a = resident_args(prog, gi, theta, false, s, rr);
                resident_terms(prog, gi, a, obs->od->K, out, rr);
                run_resident(prog, gi, a, rr.n, s);
                continue;
            }
            build_mats(prog, gi, theta, g.fwd_tasks.begin, g.fwd_tasks.end, s, rr);
            forward(prog, gi, psi + gd.psi_off, (int64_t)1 << g.n, rr.ident, s, rr);
            pauli_group(prog, gi, psi + gd.psi_off, nullptr, nullptr, obs->od->K, out, s, rr);
        }
    });
}

tq_status tq_adjoint_grad(tq_program prog, const float *theta, tq_observables obs, const float *upstream, float *grad,
                          float *expectations, void *stream)
{
    return guarded([&] {
        if (!prog || !obs) fail(TQ_E_INVALID, "program or observables is NULL");
        const ProgramData &pd = *prog->pd;
        check_obs_fit(prog, obs);
        if (pd.B == 0) return;
        if (pd.S > 0 && (!theta || !grad)) fail(TQ_E_INVALID, "symbol_values or grad is NULL");
        if (obs->od->K > 0 && !upstream) fail(TQ_E_INVALID, "upstream is NULL");
        check_align(theta, 4, "symbol_values");
        check_align(grad, 4, "grad");
        check_align(upstream, 4, "upstream");
        check_align(expectations, 4, "expectations");
        ensure_device(prog);
        ensure_obs(prog, *obs->od);
        hipStream_t s = as_stream(stream);
        float2 *psi = psi_ws(prog), *phi = phi_ws(prog);
        const int K = obs->od->K;
        for (size_t gi = 0; gi < pd.groups.size(); gi++) {
            const Group &g = *pd.groups[gi];
            GroupDev &gd = *prog->gdev[gi];
            ObsGroupDev &og = *prog->obs_dev[gi];
            const int nrows = (int)g.rows.size();
            const int64_t stride = (int64_t)1 << g.n;
            const RunRows rr = own_rows(prog, gi);
            if (resident(prog, gi, true, og.tmax)) {
                ResArgs a = resident_args(prog, gi, theta, pd.S > 0, s, rr);
                resident_terms(prog, gi, a, K, expectations, rr);
                if (pd.S > 0) {
                    a.upstream = upstream;
                    a.grad = grad;
                    a.nacc = og.tmax + g.n_gslots;
                }
                a.nacc = std::max(a.nacc, 1);
                run_resident(prog, gi, a, rr.n, s);
                continue;
            }
            build_mats(prog, gi, theta, g.fwd_tasks.begin, g.rev_tasks.end, s, rr);
            forward(prog, gi, psi + gd.psi_off, stride, rr.ident, s, rr);
            if (pd.S == 0) {
                if (expectations && K > 0)
                    pauli_group(prog, gi, psi + gd.psi_off, nullptr, nullptr, K, expectations, s, rr);
                continue;
            }
            // phi = H_g psi, with the expectations from the same sweep
            if (K > 0)
                pauli_group(prog, gi, psi + gd.psi_off, phi + gd.psi_off, upstream, K, expectations, s, rr);
            else
                hip_check(launch_zero_tail(phi + gd.psi_off, stride, (const int32_t *)gd.ident.p, nrows, 0, stride, s),
                          "phi clear");
            // reverse sweep
            const int trl = g.rev.empty() ? 0 : g.n - g.rev[0].geom.t;
            const int wg = wg_for(nrows, trl);
            double *gpart =
                (double *)prog->gpart.ensure(sizeof(double) * (size_t)nrows * wg * std::max(g.n_gslots, 1));
            int gbase = 0;
            for (size_t pi = 0; pi < g.rev.size(); pi++) {
                const Pass &ps = g.rev[pi];
                RevArgs r{};
                r.psi = psi + gd.psi_off;
                r.phi = phi + gd.psi_off;
                r.row_stride = stride;
                r.rows = (const int32_t *)gd.ident.p;
                r.mats = mat_ws(prog) + gd.mat_off;
                r.mat_stride = std::max(g.mat_block, 1);
                r.ops = (const PassOp *)gd.rev_ops.p;
                r.stages = (const Stage *)gd.rev_stages.p + gd.rev_stage_off[pi];
                r.nstages = (int)ps.stages.size();
                r.g = ps.geom;
                r.tiles_log2 = g.n - ps.geom.t;
                r.wg_per_row = wg;
                r.store = pi + 1 < g.rev.size();
                r.gpart = gpart;
                r.n_gslots = g.n_gslots;
                int gc = 0;
                for (const PassOp &op : ps.ops) gc += op.ngrad;
                r.gbase = gbase;
                r.gcount = gc;
                r.mat_begin = ps.mat_begin;
                r.mat_end = ps.mat_end;
                gbase += gc;
                // (a structure without symbolic parameters has no generated
                // reverse passes: it takes the precompiled kernel)
                if (pd.opt.specialize && g.n_gslots > 0) {
                    std::string log;
                    const hipError_t e = launch_rev_pass_spec(g, (int)pi, r, nrows, s, &log, &gd.pass_memo);
                    if (e == hipErrorInvalidSource) fail(TQ_E_DEVICE, log);
                    hip_check(e, "specialised reverse pass launch");
                    continue;
                }
                hip_check(launch_rev_pass(r, nrows, s), "reverse pass launch");
            }
            GradReduceArgs gr{};
            gr.rows = (const int32_t *)gd.rows.p;
            gr.gpart = gpart;
            gr.wg_per_row = wg;
            gr.n_gslots = g.n_gslots;
            gr.sym_begin = (const int32_t *)gd.sym_begin.p;
            gr.sym_gslots = (const int32_t *)gd.sym_gslots.p;
            gr.gslot_slot = (const int32_t *)gd.gslot_slot.p;
            gr.slot_scale = (const double *)gd.scale.p;
            gr.uniform = g.uniform_slots;
            gr.n_slots = g.n_slots;
            gr.S = pd.S;
            gr.grad = grad;
            hip_check(launch_grad_reduce(gr, nrows, s), "gradient reduce launch");
        }
    });
}

tq_status tq_observables_terms(tq_observables obs, int32_t *Kt)
{
    return guarded([&] {
        if (!obs || !Kt) fail(TQ_E_INVALID, "observables handle or Kt is NULL");
        int most = 0;
        const ObsData &od = *obs->od;
        for (int b = 0; b < od.B; b++) {
            int n = 0;
            for (int k = 0; k < od.K; k++)
                for (const HTerm &h : od.sums[(size_t)b * od.K + k]) n += !h.factors.empty();
            most = std::max(most, n);
        }
        *Kt = most;
    });
}

tq_status tq_sampled_expectation(tq_program prog, const float *theta, tq_observables obs, int32_t reps, uint64_t seed,
                                 float *out, float *term_out, void *stream)
{
    return guarded([&] {
        if (!prog || !obs) fail(TQ_E_INVALID, "program or observables is NULL");
        const ProgramData &pd = *prog->pd;
        check_obs_fit(prog, obs);
        if (reps < 1 || reps >= (1 << 24)) fail(TQ_E_INVALID, "repetitions must be in [1, 2^24)");
        const int K = obs->od->K;
        if ((int64_t)pd.B * K >= kMaxCounterRows)
            fail(TQ_E_UNSUPPORTED, "sampled expectation: B x K must be below 2^24 (the shot counter)");
        if (pd.B == 0 || K == 0) return;
        if (!out) fail(TQ_E_INVALID, "out is NULL");
        if (pd.S > 0 && !theta) fail(TQ_E_INVALID, "symbol_values is NULL");
        check_align(out, 4, "out");
        check_align(term_out, 4, "term_out");
        check_align(theta, 4, "symbol_values");
        ensure_device(prog);
        prepare_terms(obs);
        hipStream_t s = as_stream(stream);
        const int Kt = obs->Kt;
        float *tv = (float *)prog->xterm.ensure(sizeof(float) * (size_t)pd.B * std::max(Kt, 1));
        if (Kt > 0) expectations_all(prog, theta, *obs->terms, tv, s);
        SampledArgs a = sampled_args(obs, reps, seed);
        a.tv = tv;
        a.nrows = pd.B;
        a.counts = (uint32_t *)prog->xcounts.ensure(sizeof(uint32_t) * (size_t)pd.B * std::max(Kt, 1));
        a.out = out;
        hip_check(launch_sampled(a, s), "sampled expectation launch");
        if (term_out && Kt > 0)
            hip_check(hipMemcpyAsync(term_out, tv, sizeof(float) * (size_t)pd.B * Kt, hipMemcpyDeviceToDevice, s),
                      "term values copy");
    });
}

tq_status tq_param_shift_grad(tq_program prog, const float *theta, tq_observables obs, const float *upstream,
                              int32_t reps, uint64_t seed, float *grad, void *stream)
{
    return guarded([&] {
        if (!prog || !obs) fail(TQ_E_INVALID, "program or observables is NULL");
        const ProgramData &pd = *prog->pd;
        check_obs_fit(prog, obs);
        if (reps < 0 || reps >= (1 << 24)) fail(TQ_E_INVALID, "repetitions must be in [0, 2^24)");
        if (pd.B == 0 || pd.S == 0) return;
        if (!theta || !grad) fail(TQ_E_INVALID, "symbol_values or grad is NULL");
        if (obs->od->K > 0 && !upstream) fail(TQ_E_INVALID, "upstream is NULL");
        check_align(theta, 4, "symbol_values");
        check_align(grad, 4, "grad");
        check_align(upstream, 4, "upstream");
        for (auto &gp : pd.groups)
            for (const Occurrence &oc : gp->occurrences) {
                double delta, factor;
                if (!shift_rule(oc.blob_op, oc.param, &delta, &factor))
                    fail(TQ_E_UNSUPPORTED, "parameter shift: a symbolic parameter has no two-term shift rule "
                                           "(fSim theta; use the adjoint or finite differences)");
            }
        ensure_device(prog);
        shift_grad(prog, theta, obs, upstream, kParamShift, reps, seed, 0.0, grad, as_stream(stream));
    });
}

tq_status tq_finite_diff_grad(tq_program prog, const float *theta, tq_observables obs, const float *upstream,
                              double eps, float *grad, void *stream)
{
    return guarded([&] {
        if (!prog || !obs) fail(TQ_E_INVALID, "program or observables is NULL");
        const ProgramData &pd = *prog->pd;
        check_obs_fit(prog, obs);
        if (!(eps > 0.0) || !(eps < 1e300)) fail(TQ_E_INVALID, "eps must be a finite number > 0");
        if (pd.B == 0 || pd.S == 0) return;
        if (!theta || !grad) fail(TQ_E_INVALID, "symbol_values or grad is NULL");
        if (obs->od->K > 0 && !upstream) fail(TQ_E_INVALID, "upstream is NULL");
        check_align(theta, 4, "symbol_values");
        check_align(grad, 4, "grad");
        check_align(upstream, 4, "upstream");
        ensure_device(prog);
        shift_grad(prog, theta, obs, upstream, kFiniteDiff, 0, 0, eps, grad, as_stream(stream));
    });
}

tq_status tq_sample(tq_program prog, const float *theta, int64_t n_shots, uint64_t seed, uint64_t *out, void *stream)
{
    return tq_sample_with_amplitudes(prog, theta, n_shots, seed, out, nullptr, 0, nullptr, stream);
}

tq_status tq_sample_with_amplitudes(tq_program prog, const float *theta, int64_t n_shots, uint64_t seed, uint64_t *out,
                                    const uint64_t *bitstrings, int64_t M, void *amps, void *stream)
{
    return guarded([&] {
        if (!prog) fail(TQ_E_INVALID, "program is NULL");
        if (n_shots < 0) fail(TQ_E_INVALID, "n_shots is negative");
        if (M < 0) fail(TQ_E_INVALID, "M is negative");
        const ProgramData &pd = *prog->pd;
        if (pd.B == 0 || (n_shots == 0 && M == 0)) return;
        if (n_shots > 0 && !out) fail(TQ_E_INVALID, "out is NULL");
        if (M > 0 && (!bitstrings || !amps)) fail(TQ_E_INVALID, "bitstrings or amps is NULL");
        if (pd.S > 0 && !theta) fail(TQ_E_INVALID, "symbol_values is NULL");
        check_align(out, 8, "out");
        check_align(bitstrings, 8, "bitstrings");
        check_align(amps, 8, "amps");
        check_align(theta, 4, "symbol_values");
        ensure_device(prog);
        hipStream_t s = as_stream(stream);
        float2 *psi = psi_ws(prog);
        for (size_t gi = 0; gi < pd.groups.size(); gi++) {
            const Group &g = *pd.groups[gi];
            GroupDev &gd = *prog->gdev[gi];
            forward_to_ws(prog, gi, theta, psi + gd.psi_off, s, own_rows(prog, gi));
            if (M > 0) {
                GatherArgs ga{};
                ga.state = psi + gd.psi_off;
                ga.row_stride = (int64_t)1 << g.n;
                ga.rows = (const int32_t *)gd.ident.p;
                ga.brows = (const int32_t *)gd.rows.p;
                ga.n = g.n;
                ga.bits = bitstrings;
                ga.M = M;
                ga.out = (float2 *)amps;
                hip_check(launch_gather(ga, (int)g.rows.size(), s), "gather launch");
            }
            if (n_shots == 0) continue;
            SampArgs a{};
            a.state = psi + gd.psi_off;
            a.row_stride = (int64_t)1 << g.n;
            a.vec16 = g.n >= 1;  // workspace rows are 512-byte aligned, 2^n amplitudes apart
            a.rows = (const int32_t *)gd.ident.p;
            a.brows = (const int32_t *)gd.rows.p;
            fill_levels(a, g.n);
            a.levels = (uint64_t *)prog->levels.ensure(sizeof(uint64_t) * a.row_level * g.rows.size());
            a.n_shots = n_shots;
            a.seed = seed;
            a.out = out;
            hip_check(launch_sample(a, (int)g.rows.size(), s), "sampler launch");
        }
    });
}

tq_status tq_amplitudes(tq_program prog, const float *theta, const uint64_t *bitstrings, int64_t M, void *amps,
                        void *stream)
{
    return guarded([&] {
        if (!prog) fail(TQ_E_INVALID, "program is NULL");
        if (M < 0) fail(TQ_E_INVALID, "M is negative");
        const ProgramData &pd = *prog->pd;
        if (pd.B == 0 || M == 0) return;
        if (!bitstrings || !amps) fail(TQ_E_INVALID, "bitstrings or amps is NULL");
        if (pd.S > 0 && !theta) fail(TQ_E_INVALID, "symbol_values is NULL");
        check_align(bitstrings, 8, "bitstrings");
        check_align(amps, 8, "amps");
        check_align(theta, 4, "symbol_values");
        ensure_device(prog);
        hipStream_t s = as_stream(stream);
        float2 *psi = psi_ws(prog);
        for (size_t gi = 0; gi < pd.groups.size(); gi++) {
            const Group &g = *pd.groups[gi];
            GroupDev &gd = *prog->gdev[gi];
            forward_to_ws(prog, gi, theta, psi + gd.psi_off, s, own_rows(prog, gi));
            GatherArgs a{};
            a.state = psi + gd.psi_off;
            a.row_stride = (int64_t)1 << g.n;
            a.rows = (const int32_t *)gd.ident.p;
            a.brows = (const int32_t *)gd.rows.p;
            a.n = g.n;
            a.bits = bitstrings;
            a.M = M;
            a.out = (float2 *)amps;
            hip_check(launch_gather(a, (int)g.rows.size(), s), "gather launch");
        }
    });
}

tq_status tq_sample_from_state(const void *states, int32_t B, int32_t n, int64_t n_shots, uint64_t seed,
                               uint64_t *out, void *stream)
{
    return guarded([&] {
        if (B < 0 || n < 0 || n > kMaxQubits || n_shots < 0) fail(TQ_E_INVALID, "bad B, n or n_shots");
        if (B == 0 || n_shots == 0) return;
        if (!states || !out) fail(TQ_E_INVALID, "states or out is NULL");
        check_align(states, 8, "states");
        check_align(out, 8, "out");
        hipStream_t s = as_stream(stream);
        SampArgs a{};
        a.state = (const float2 *)states;
        a.row_stride = (int64_t)1 << n;
        a.vec16 = reinterpret_cast<uintptr_t>(states) % 16 == 0 && n >= 1;
        fill_levels(a, n);
        // stream-ordered workspace: allocated and released in the stream's order
        void *lv = nullptr;
        if (hipMallocAsync(&lv, sizeof(uint64_t) * a.row_level * (size_t)B, s) != hipSuccess) {
            (void)hipGetLastError();
            fail(TQ_E_NOMEM, "sampler workspace allocation failed");
        }
        a.levels = (uint64_t *)lv;
        a.n_shots = n_shots;
        a.seed = seed;
        a.out = out;
        hipError_t e = launch_sample(a, B, s);
        hipError_t f = hipFreeAsync(lv, s);
        hip_check(e, "sampler launch");
        hip_check(f, "hipFreeAsync");
    });
}

tq_status tq_sample_from_state_noalloc(const void *states, int32_t B, int32_t n, int64_t n_shots, uint64_t seed,
                                       uint64_t *out, void *stream)
{
    return guarded([&] {
        if (B < 0 || n < 0 || n > kMaxQubits || n_shots < 0) fail(TQ_E_INVALID, "bad B, n or n_shots");
        if (B == 0 || n_shots == 0) return;
        if (!states || !out) fail(TQ_E_INVALID, "states or out is NULL");
        check_align(states, 8, "states");
        check_align(out, 8, "out");
        SampArgs a{};
        a.state = (const float2 *)states;
        a.row_stride = (int64_t)1 << n;
        a.vec16 = reinterpret_cast<uintptr_t>(states) % 16 == 0 && n >= 1;
        fill_levels(a, n);
        if ((int64_t)B * a.row_level > kStaticLevelEntries)
            fail(TQ_E_UNSUPPORTED, "tq_sample_from_state_noalloc: B * (level entries per row) = " +
                                       std::to_string((int64_t)B * a.row_level) + " exceeds its static workspace of " +
                                       std::to_string(kStaticLevelEntries) + " entries (about B 2^n / 63 <= 2^22)");
        uint64_t *lv = nullptr;
        hip_check(static_levels(&lv), "static sampler workspace lookup");
        // every level entry is written (level 1 from the state, the others
        // from the level below) before it is read: nothing to clear
        a.levels = lv;
        a.n_shots = n_shots;
        a.seed = seed;
        a.out = out;
        hip_check(launch_sample(a, B, as_stream(stream)), "sampler launch");
    });
}

tq_status tq_amplitudes_from_state(const void *states, int32_t B, int32_t n, const uint64_t *bitstrings, int64_t M,
                                   void *amps, void *stream)
{
    return guarded([&] {
        if (B < 0 || n < 0 || n > kMaxQubits || M < 0) fail(TQ_E_INVALID, "bad B, n or M");
        if (B == 0 || M == 0) return;
        if (!states || !bitstrings || !amps) fail(TQ_E_INVALID, "states, bitstrings or amps is NULL");
        check_align(states, 8, "states");
        check_align(bitstrings, 8, "bitstrings");
        check_align(amps, 8, "amps");
        GatherArgs a{};
        a.state = (const float2 *)states;
        a.row_stride = (int64_t)1 << n;
        a.n = n;
        a.bits = bitstrings;
        a.M = M;
        a.out = (float2 *)amps;
        hip_check(launch_gather(a, B, as_stream(stream)), "gather launch");
    });
}

tq_status tq_build_matrices(tq_program prog, const float *theta, void *out, int64_t cap, int64_t *entries, void *stream)
{
    return guarded([&] {
        if (!prog) fail(TQ_E_INVALID, "program is NULL");
        const ProgramData &pd = *prog->pd;
        int64_t total = 0;
        for (auto &gp : pd.groups) total += (int64_t)gp->rows.size() * std::max(gp->mat_block, 1);
        if (entries) *entries = total;
        if (!out) return;
        if (cap < total) fail(TQ_E_INVALID, "out holds fewer than the needed entries");
        if (pd.S > 0 && !theta) fail(TQ_E_INVALID, "symbol_values is NULL");
        check_align(out, 16, "out");
        ensure_device(prog);
        hipStream_t s = as_stream(stream);
        int64_t off = 0;
        for (size_t gi = 0; gi < pd.groups.size(); gi++) {
            const Group &g = *pd.groups[gi];
            GroupDev &gd = *prog->gdev[gi];
            build_mats(prog, gi, theta, g.fwd_tasks.begin, g.rev_tasks.end, s, own_rows(prog, gi));
            const size_t n = g.rows.size() * (size_t)std::max(g.mat_block, 1);
            hip_check(hipMemcpyAsync((double2 *)out + off, mat_ws(prog) + gd.mat_off, n * sizeof(double2),
                                     hipMemcpyDeviceToDevice, s),
                      "matrix copy");
            off += (int64_t)n;
        }
    });
}

tq_status tq_gate_matrix(int32_t op, const double *params, const double *explicit_m, int32_t cblock, int32_t deriv,
                         int32_t which, double *out, int32_t *dim, double *phase)
{
    return guarded([&] {
        if (!out || !dim || !phase) fail(TQ_E_INVALID, "out, dim or phase is NULL");
        if (op < 1 || op >= OP_COUNT) fail(TQ_E_INVALID, "unknown opcode");
        const bool expl = op == OP_MATRIX1 || op == OP_MATRIX2;
        if (expl && !explicit_m) fail(TQ_E_INVALID, "explicit matrix is NULL");
        double eta[3] = {params ? params[0] : 0.0, params ? params[1] : 0.0, 0.0};
        const int form = cblock && (op == OP_CNOT || op == OP_CNOTPOW) ? FORM_CBLOCK : FORM_FULL;
        const int d = gate_table_host(op, eta, explicit_m, form, deriv ? 1 : 0, which, out);
        if (d == 0) fail(TQ_E_INVALID, deriv ? "the gate has no derivative" : "unknown opcode");
        *dim = d;
        *phase = gate_left_out_phase(op, eta[0]);
    });
}

tq_status tq_profile_start(const char *kernel)
{
    return guarded([&] { profile_start(kernel); });
}

tq_status tq_profile_read(int64_t *launches, double *total_ms)
{
    return guarded([&] {
        if (!launches || !total_ms) fail(TQ_E_INVALID, "launches or total_ms is NULL");
        hip_check(profile_read(launches, total_ms), "profile read");
    });
}

tq_status tq_program_describe(tq_program prog, char *buf, size_t cap, size_t *needed)
{
    return guarded([&] {
        if (!prog) fail(TQ_E_INVALID, "program is NULL");
        const ProgramData &pd = *prog->pd;
        std::ostringstream o;
        static const char *kinds[] = {"?", "M1", "M2", "D1", "D2", "P2", "F2"};
        o << "{\"B\":" << pd.B << ",\"S\":" << pd.S << ",\"nmax\":" << pd.nmax << ",\"tile\":" << pd.opt.tile
          << ",\"low\":" << pd.opt.low << ",\"groups\":[";
        for (size_t gi = 0; gi < pd.groups.size(); gi++) {
            const Group &g = *pd.groups[gi];
            std::map<int32_t, int> members_at;  // matrix offset -> member count
            for (const BuildTask &bt : g.tasks)
                if (bt.kind != BT_DERIV) members_at[bt.out] = bt.mem_count;
            int absorbed = 0;
            for (int q = 0; q < g.n; q++)
                for (const BuildTask &bt : g.tasks)
                    if (bt.out == g.init_mat[q]) absorbed += bt.mem_count;
            o << (gi ? "," : "") << "{\"n\":" << g.n << ",\"rows\":" << g.rows.size() << ",\"gates\":" << g.gates.size()
              << ",\"row_ids\":[";
            for (size_t r = 0; r < g.rows.size(); r++) o << (r ? "," : "") << g.rows[r];
            o << "],\"init_mat\":[";
            for (int q = 0; q < g.n; q++) o << (q ? "," : "") << g.init_mat[q];
            // build tasks: kind (0 product, 1 dagger, 2 derivative), dim, storage
            // (0 dense, 1 diagonal, 2 / 3 the (a, b) pair of a I + b XX / YY, 4 the
            // six entries of an excitation-preserving 4x4), parameter, offset in the
            // row block, members [gate, qubit order swapped, controlled block]
            o << "],\"tasks\":[";
            for (size_t t = 0; t < g.tasks.size(); t++) {
                const BuildTask &bt = g.tasks[t];
                o << (t ? "," : "") << "[" << (int)bt.kind << "," << (int)bt.dim << "," << (int)bt.diag << ","
                  << (int)bt.which << "," << bt.out << ",[";
                for (int m = 0; m < bt.mem_count; m++) {
                    const Member &mb = g.members[bt.mem_begin + m];
                    o << (m ? "," : "") << "[" << mb.gate << "," << (int)mb.swapped << "," << (int)mb.form << "]";
                }
                o << "]]";
            }
            o << "]";
            o
              << ",\"slots\":" << g.n_slots << ",\"mat_block\":" << g.mat_block << ",\"n_gslots\":" << g.n_gslots
              << ",\"absorbed\":" << absorbed << ",\"uniform_slots\":" << (g.uniform_slots ? 1 : 0);
            // symbolic blob parameters (what the parameter-shift rule moves):
            // [slot, second slot or -1, symbol, blob opcode, parameter index]
            o << ",\"occurrences\":[";
            for (size_t k = 0; k < g.occurrences.size(); k++) {
                const Occurrence &oc = g.occurrences[k];
                o << (k ? "," : "") << "[" << oc.slot[0] << "," << oc.slot[1] << "," << oc.sym << ","
                  << oc.blob_op << "," << (int)oc.param << "]";
            }
            o << "]";
            // the observables last used with the program: Z-only stream, and the
            // terms of each generated expectation pass and H_g pass
            if (gi < prog->obs_dev.size()) {
                const ObsGroupDev &og = *prog->obs_dev[gi];
                o << ",\"obs\":{\"diag\":" << (og.diag ? 1 : 0);
                // (expectation passes of every observable set, in order)
                std::vector<size_t> exp_terms, phi_terms;
                for (const ObsGroupDev::SpecSet &set : og.spec_sets)
                    for (const PauliPass &pp : set.passes) exp_terms.push_back(pp.terms.size());
                for (const PauliPass &pp : og.phi_passes) phi_terms.push_back(pp.terms.size());
                for (int v = 0; v < 2; v++) {
                    const std::vector<size_t> &pt = v == 0 ? exp_terms : phi_terms;
                    o << (v == 0 ? ",\"exp_passes\":[" : ",\"phi_passes\":[");
                    for (size_t k = 0; k < pt.size(); k++) o << (k ? "," : "") << pt[k];
                    o << "]";
                }
                o << ",\"exp_sets\":" << og.spec_sets.size();
                o << "}";
            }
            for (int dir = 0; dir < 2; dir++) {
                const std::vector<Pass> &pv = dir == 0 ? g.fwd : g.rev;
                o << (dir == 0 ? ",\"fwd\":[" : ",\"rev\":[");
                for (size_t pi = 0; pi < pv.size(); pi++) {
                    const Pass &ps = pv[pi];
                    o << (pi ? "," : "") << "{\"t\":" << ps.geom.t << ",\"c\":" << ps.geom.c << ",\"h\":" << ps.geom.h
                      << ",\"hb\":[";
                    for (int k = 0; k < ps.geom.h; k++) o << (k ? "," : "") << (int)ps.geom.hb[k];
                    o << "],\"product_init\":" << (ps.product_init ? 1 : 0) << ",\"ops\":[";
                    for (size_t k = 0; k < ps.ops.size(); k++) {
                        const PassOp &op = ps.ops[k];
                        o << (k ? "," : "") << "{\"kind\":\"" << kinds[op.kind] << "\",\"p\":[" << (int)op.p0 << ","
                          << (int)op.p1 << "],\"l\":[" << (int)op.l0 << "," << (int)op.l1 << "],\"ctrl\":" << (int)op.ctrl
                          << ",\"hint\":" << (int)op.hint
                          << ",\"ngrad\":" << (int)op.ngrad << ",\"members\":"
                          << (members_at.count(op.mat) ? members_at[op.mat] : 0);
                        if (dir == 1) {  // generator terms [x, z, ny, c] of each gradient parameter
                            o << ",\"gen\":[";
                            for (int j = 0; j < op.ngrad; j++) {
                                std::vector<GenTerm> gt;
                                o << (j ? "," : "") << "[";
                                if (op_generator(g, op, j, &gt))
                                    for (size_t m = 0; m < gt.size(); m++)
                                        o << (m ? "," : "") << "[" << (int)gt[m].x << "," << (int)gt[m].z << ","
                                          << (int)gt[m].ny << "," << std::setprecision(17) << gt[m].c << "]";
                                o << "]";
                            }
                            o << "]";
                        }
                        o << "}";
                    }
                    o << "],\"stages\":[";
                    for (size_t k = 0; k < ps.stages.size(); k++) {
                        const Stage &sg = ps.stages[k];
                        o << (k ? "," : "") << "{\"r\":" << (int)sg.r << ",\"bits\":[";
                        for (int j = 0; j < sg.r; j++) o << (j ? "," : "") << (int)sg.bits[j];
                        o << "],\"ops\":" << (sg.op_end - sg.op_begin) << ",\"dense\":" << (int)sg.dense << "}";
                    }
                    o << "]}";
                }
                o << "]";
            }
            o << "}";
        }
        o << "]}";
        const std::string js = o.str();
        if (needed) *needed = js.size() + 1;
        if (buf && cap > 0) {
            size_t n = std::min(cap - 1, js.size());
            std::memcpy(buf, js.data(), n);
            buf[n] = 0;
        }
    });
}

} // extern "C"
