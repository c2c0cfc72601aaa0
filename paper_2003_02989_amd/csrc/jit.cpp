// jit.cpp -- generation, run-time compilation and launch of kernels
// specialised for one circuit structure: the resident-circuit kernel and the
// forward and reverse tile passes.  The generated code calls the same
// register-op templates (device_ops.h) the precompiled kernels dispatch to,
// with the register bits, tile bits and matrix offsets of every op and stage
// written in as constants; the parts around the stages (tile loads and
// stores, product-state generation, expectations, reductions) are the
// precompiled kernels' own device functions.
#include "jit.h"

#include "kernels.h"

#include <hip/hiprtc.h>

#include <algorithm>
#include <tuple>
#include <cmath>
#include <array>
#include <cstdio>
#include <map>
#include <memory>
#include <mutex>
#include <set>
#include <cstring>
#include <sstream>
#include <vector>
#include <atomic>
#include <cstdlib>
#include <fstream>
#include <iterator>
#include <thread>
#include <sys/stat.h>
#include <unistd.h>

namespace tq {
namespace {

// tq_internal.h, kernel_args.h and device_ops.h as one text (written by the
// build from the headers, with their local includes removed)
const char kPrelude[] =
#include "jit_prelude.inc"
    ;

std::string N(long v) { return std::to_string(v); }
// a double literal that reads back exactly
std::string dbl(double v)
{
    char b[40];
    snprintf(b, sizeof b, "%.17g", v);
    return std::string(b).find_first_of(".en") == std::string::npos ? std::string(b) + ".0" : std::string(b);
}

// LDS of a specialised Pauli pass: the tile, its high-bit offsets and the
// per-wave sums of at most `nk` observables (every pass has at most 16)
int pauli_spec_threads(const TileGeom &g) { return 1 << (g.t - 4); }
size_t pauli_spec_lds_bytes(const TileGeom &g, int K)
{
    // the tile, its high-bit offsets, and per-wave sums of the observables
    // (at least 16 x 16 slots)
    const size_t waves = (size_t)pauli_spec_threads(g) / 64;
    return sizeof(float2) * ((size_t)1 << g.t) + sizeof(uint64_t) * ((size_t)1 << g.h) +
           sizeof(double) * std::max<size_t>(16 * 16, waves * (size_t)K);
}

uint32_t host_sw(uint32_t i) { return i ^ ((i >> 5) & 31u); }

// Where a kernel's stage code finds its data.
struct Env {
    int t;          // tile bits: a stage of r register bits has 2^(t - r) items
    int mbase;      // op matrix offsets are taken relative to this
    std::string G;  // base of dense stage matrices (absolute offsets)
    bool fixed;     // the tile has fixed bits: a bit outside it reads fb
    // reverse stages: accumulator of gradient slot s is acc[(tid >> 6) * stride + s + shift]
    std::string acc_stride;
    std::string acc_shift;
    // reverse tile passes with few gradient slots: each thread's partial sum
    // of slot s stays in register gacc_[s + gshift] over all its tiles (one
    // wavefront sum per slot at the end of the kernel instead of one per
    // stage and tile)
    bool gacc_reg = false;
    int gshift = 0;
    // forward tile passes: the phase classes of the pass's diagonal runs, in
    // the order the stages meet them (see cut_classes), and the next to use
    const std::vector<struct CutClass> *cuts = nullptr;
    mutable size_t cut_next = 0;
    int nt = kThreads;  // threads of the workgroup
    const Group *grp = nullptr;  // reverse stages: gradients from gate generators where known
    const Group *fgrp = nullptr; // forward stages: constant single-qubit ops written out (const_m1)
    // keep each op's matrix reads next to the op (opaque per-item offset,
    // scheduling barriers between reverse ops): needed where registers are
    // short (tile passes, four waves per SIMD)
    bool pin = true;
};

// An op bit at tile position l (global position p): from the item's base
// index, or from the tile's fixed bits.
std::string bit(const Env &e, uint8_t l, uint8_t p)
{
    if (l != kFixed) return "((base >> " + N(l) + ") & 1u)";
    return e.fixed ? "((uint32_t)(fb >> " + N(p) + ") & 1u)" : std::string("0u");
}
std::string ent(int mat) { return "M[z_ + " + N(mat) + "]"; }

// The call of rd1/rd2/rscale (or its _dot form) for a diagonal op with
// matrix offset `mat` on register array `v`.
std::string diag_call(const Env &e, const PassOp &op, int R, int mat, bool dot, const std::string &v)
{
    const std::string sfx = dot ? "_dot" : "", args = dot ? "v, f" : v;
    const std::string Rs = N(R);
    // entries exactly 1 in W (skipped) are exactly 0 in dW (skipped in dots)
    const int um = op.hint & 0xf;
    const std::string ux = um ? (dot ? "_dotz" : "u") : sfx;
    const std::string ut = um ? ", " + N(um) : "";
    if (op.kind == K_D1) {
        if (op.s0 != kFixed)
            return "rd1" + ux + "<" + Rs + ", " + N(op.s0) + ut + ">(" + args + ", " + ent(mat) + ", " + ent(mat + 1) + ")";
        return "rscale" + sfx + "<" + Rs + ">(" + args + ", zsel(" + bit(e, op.l0, op.p0) + ", " + ent(mat) + ", " +
               ent(mat + 1) + "))";
    }
    const bool r0 = op.s0 != kFixed, r1 = op.s1 != kFixed;
    if (r0 && r1) {
        const int j0 = std::min(op.s0, op.s1), j1 = std::max(op.s0, op.s1);
        const bool q0lo = op.s0 < op.s1;
        const int x[4] = {0, q0lo ? 1 : 2, q0lo ? 2 : 1, 3};
        // the unit mask in the register-bit order of the arguments
        int um2 = 0;
        for (int k = 0; k < 4; k++)
            if ((um >> x[k]) & 1) um2 |= 1 << k;
        const std::string ut2 = um ? ", " + N(um2) : "";
        return "rd2" + ux + "<" + Rs + ", " + N(j0) + ", " + N(j1) + ut2 + ">(" + args + ", " + ent(mat + x[0]) + ", " +
               ent(mat + x[1]) + ", " + ent(mat + x[2]) + ", " + ent(mat + x[3]) + ")";
    }
    if (r0) {  // entries (v, 2 + v) with v the bit of q1
        const std::string b = bit(e, op.l1, op.p1);
        return "rd1" + sfx + "<" + Rs + ", " + N(op.s0) + ">(" + args + ", zsel(" + b + ", " + ent(mat) + ", " +
               ent(mat + 1) + "), zsel(" + b + ", " + ent(mat + 2) + ", " + ent(mat + 3) + "))";
    }
    if (r1) {  // entries (2v, 2v + 1) with v the bit of q0
        const std::string b = bit(e, op.l0, op.p0);
        return "rd1" + sfx + "<" + Rs + ", " + N(op.s1) + ">(" + args + ", zsel(" + b + ", " + ent(mat) + ", " +
               ent(mat + 2) + "), zsel(" + b + ", " + ent(mat + 1) + ", " + ent(mat + 3) + "))";
    }
    const std::string b0 = bit(e, op.l0, op.p0), b1 = bit(e, op.l1, op.p1);
    return "rscale" + sfx + "<" + Rs + ">(" + args + ", zsel(" + b0 + ", zsel(" + b1 + ", " + ent(mat) + ", " +
           ent(mat + 1) + "), zsel(" + b1 + ", " + ent(mat + 2) + ", " + ent(mat + 3) + ")))";
}

// op applied to register array `v` (matrix at offset mat)
std::string apply(const Env &e, const PassOp &op, int R, int mat, const std::string &v)
{
    const std::string Rs = N(R), m = "M + (z_ + " + N(mat) + ")";
    if (op.kind == K_M1 && (op.hint & kHintX)) {  // a swap: no matrix read, no arithmetic
        if (!op.ctrl) return "rx1<" + Rs + ", " + N(op.s0) + ">(" + v + ");";
        if (op.s1 != kFixed) return "rx1c<" + Rs + ", " + N(op.s0) + ", " + N(op.s1) + ">(" + v + ");";
        return "rx1_if<" + Rs + ", " + N(op.s0) + ">(" + v + ", " + bit(e, op.l1, op.p1) + " == " + N(op.cval) + "u);";
    }
    switch (op.kind) {
    case K_M1:
        if (!op.ctrl && (op.hint & kHintReal)) return "rm1r<" + Rs + ", " + N(op.s0) + ">(" + v + ", " + m + ");";
        if (!op.ctrl && (op.hint & kHintRX)) return "rm1x<" + Rs + ", " + N(op.s0) + ">(" + v + ", " + m + ");";
        if (!op.ctrl) return "rm1<" + Rs + ", " + N(op.s0) + ">(" + v + ", " + m + ");";
        if (op.s1 != kFixed) return "rm1c<" + Rs + ", " + N(op.s0) + ", " + N(op.s1) + ">(" + v + ", " + m + ");";
        return "rm1_on<" + Rs + ", " + N(op.s0) + ">(" + v + ", " + m + ", " + bit(e, op.l1, op.p1) + " == " +
               N(op.cval) + "u);";
    case K_M2: return "rm2<" + Rs + ", " + N(op.s0) + ", " + N(op.s1) + ">(" + v + ", " + m + ");";
    case K_F2:
        if (op.hint & kHintSwap)
            return "rf2s<" + Rs + ", " + N(op.s0) + ", " + N(op.s1) + ", " + N(op.hint & 9) + ">(" + v + ", " + m + ");";
        if (op.hint & (9 | kHintRX))
            return "rf2x<" + Rs + ", " + N(op.s0) + ", " + N(op.s1) + ", " + N(op.hint & 9) + ", " +
                   ((op.hint & kHintRX) ? "true" : "false") + ">(" + v + ", " + m + ");";
        return "rf2<" + Rs + ", " + N(op.s0) + ", " + N(op.s1) + ">(" + v + ", " + m + ");";
    case K_P2:
        return std::string((op.hint & kHintRX) ? "rp2x<" : "rp2<") + Rs + ", " + N(std::min(op.s0, op.s1)) + ", " +
               N(std::max(op.s0, op.s1)) + ">(" + v + ", " + ent(mat) + ", " + ent(mat + 1) + ", " +
               (op.ptype == 2 ? "-1.0" : "1.0") + ");";
    default: return diag_call(e, op, R, mat, false, v) + ";";
    }
}

// sum of Re(conj(f) dW v) for the derivative matrix at offset d
std::string dot(const Env &e, const PassOp &op, int R, int d)
{
    const std::string Rs = N(R), m = "M + (z_ + " + N(d) + ")";
    switch (op.kind) {
    case K_M1:
        if (!op.ctrl && (op.hint & kHintReal)) return "rm1r_dot<" + Rs + ", " + N(op.s0) + ">(v, f, " + m + ")";
        if (!op.ctrl) return "rm1_dot<" + Rs + ", " + N(op.s0) + ">(v, f, " + m + ")";
        if (op.s1 != kFixed) return "rm1c_dot<" + Rs + ", " + N(op.s0) + ", " + N(op.s1) + ">(v, f, " + m + ")";
        // an item whose control is off sees the identity and a zero derivative
        return "(" + bit(e, op.l1, op.p1) + " == " + N(op.cval) + "u ? rm1_dot<" + Rs + ", " + N(op.s0) +
               ">(v, f, " + m + ") : 0.0)";
    case K_M2: return "rm2_dot<" + Rs + ", " + N(op.s0) + ", " + N(op.s1) + ">(v, f, " + m + ")";
    case K_F2: return "rf2_dot<" + Rs + ", " + N(op.s0) + ", " + N(op.s1) + ">(v, f, " + m + ")";
    case K_P2:
        return "rp2_dot<" + Rs + ", " + N(std::min(op.s0, op.s1)) + ", " + N(std::max(op.s0, op.s1)) + ">(v, f, " +
               ent(d) + ", " + ent(d + 1) + ", " + (op.ptype == 2 ? "-1.0" : "1.0") + ")";
    default: return diag_call(e, op, R, d, true, "v");
    }
}

// Im<f| G |v> for the generator terms of one parameter, on the registers
// before the op is applied, as a block that adds it to `acc`; "" when a term
// flips a bit outside the stage.  Term c i^ny X^x Z^z pairs register k with
// k' = k ^ x and contributes c (-1)^|z & bits(k')| Im(i^ny conj(f_k) v_k'),
// i.e. +-c times Im or Re of conj(f_k) v_k'.  Signs of z bits outside the
// stage are per item: the coefficients of a (k, k', part) entry are kept
// for the four values of the op's two bits, entries with proportional
// coefficient vectors share an accumulator (two FMAs per entry), and each
// accumulator is weighted once per item.
std::string gen_dot(const Env &e, const PassOp &op, int R, const std::vector<GenTerm> &terms, const std::string &acc)
{
    const int NR = 1 << R;
    const bool r0 = op.s0 != kFixed, r1 = op.s1 != kFixed;
    std::map<std::tuple<int, int, int>, std::array<double, 4>> ent;  // (k, k', re) -> coefficient per (b0, b1)
    for (const GenTerm &tm : terms) {
        // an identity term adds c Im<f|v>, which vanishes: f and v have been
        // transformed by the same unitaries since f = H_g v (H_g Hermitian),
        // so <f|v> = <psi|H_g|psi> is real
        if (tm.x == 0 && tm.z == 0) continue;
        int xr = 0;
        if (tm.x & 1) {
            if (!r0) return "";
            xr |= 1 << op.s0;
        }
        if (tm.x & 2) {
            if (!r1) return "";
            xr |= 1 << op.s1;
        }
        const int rt = ((tm.z & 1) && !r0 ? 1 : 0) | ((tm.z & 2) && !r1 ? 2 : 0);  // z bits read per item
        const double sny = (tm.ny & 2) ? -1.0 : 1.0;                              // i^2 = -1
        for (int k = 0; k < NR; k++) {
            const int kp = k ^ xr;
            int par = 0;
            if ((tm.z & 1) && r0) par ^= (kp >> op.s0) & 1;
            if ((tm.z & 2) && r1) par ^= (kp >> op.s1) & 1;
            auto it = ent.find({k, kp, tm.ny & 1});
            if (it == ent.end()) it = ent.emplace(std::make_tuple(k, kp, tm.ny & 1), std::array<double, 4>{}).first;
            for (int rho = 0; rho < 4; rho++)
                it->second[rho] += tm.c * sny * (((par ^ __builtin_popcount(rt & rho)) & 1) ? -1.0 : 1.0);
        }
    }
    // accumulator classes: coefficient vectors up to sign
    std::vector<std::array<double, 4>> cls;
    std::vector<std::vector<std::pair<std::tuple<int, int, int>, double>>> mem;
    for (auto &en : ent) {
        const std::array<double, 4> &a = en.second;
        int first = -1;
        for (int r = 0; r < 4 && first < 0; r++)
            if (std::fabs(a[r]) > 1e-15) first = r;
        if (first < 0) continue;
        const double sg = a[first] < 0 ? -1.0 : 1.0;
        std::array<double, 4> key;
        for (int r = 0; r < 4; r++) key[r] = sg * a[r];
        size_t ci = 0;
        for (; ci < cls.size(); ci++) {
            bool same = true;
            for (int r = 0; r < 4; r++) same &= std::fabs(cls[ci][r] - key[r]) <= 1e-12 * std::fabs(key[first]);
            if (same) break;
        }
        if (ci == cls.size()) {
            cls.push_back(key);
            mem.emplace_back();
        }
        mem[ci].emplace_back(en.first, sg);
    }
    // two chains per accumulator (the two FMAs of an entry), summed at the end
    std::ostringstream o;
    o << "{ ";
    for (size_t ci = 0; ci < cls.size(); ci++) o << "double t" << ci << "a = 0.0, t" << ci << "b = 0.0; ";
    for (size_t ci = 0; ci < cls.size(); ci++)
        for (auto &m : mem[ci]) {
            const int k = std::get<0>(m.first), kp = std::get<1>(m.first);
            const bool re = std::get<2>(m.first);
            const std::string p = m.second < 0 ? "-" : "", q = m.second < 0 ? "" : "-";
            const std::string A = "t" + N((long)ci) + "a", B = "t" + N((long)ci) + "b";
            const std::string F = "f[" + N(k) + "]", V = "v[" + N(kp) + "]";
            if (re)  // Re(conj(f) v) = f.x v.x + f.y v.y
                o << A << " = fma(" << p << F << ".x, " << V << ".x, " << A << "); " << B << " = fma(" << p << F
                  << ".y, " << V << ".y, " << B << "); ";
            else     // Im(conj(f) v) = f.x v.y - f.y v.x
                o << A << " = fma(" << p << F << ".x, " << V << ".y, " << A << "); " << B << " = fma(" << q << F
                  << ".y, " << V << ".x, " << B << "); ";
        }
    const std::string b0 = r0 ? "" : bit(e, op.l0, op.p0), b1 = r1 ? "" : bit(e, op.l1, op.p1);
    o << acc << " += 0.0";
    for (size_t ci = 0; ci < cls.size(); ci++) {
        const std::array<double, 4> &a = cls[ci];
        const bool v0 = a[0] != a[1] || a[2] != a[3], v1 = a[0] != a[2] || a[1] != a[3];
        std::string w;
        if (!v0 && !v1) w = dbl(a[0]);
        else if (!v1) w = "(" + b0 + " ? " + dbl(a[1]) + " : " + dbl(a[0]) + ")";
        else if (!v0) w = "(" + b1 + " ? " + dbl(a[2]) + " : " + dbl(a[0]) + ")";
        else
            w = "(" + b1 + " ? (" + b0 + " ? " + dbl(a[3]) + " : " + dbl(a[2]) + ") : (" + b0 + " ? " + dbl(a[1]) +
                " : " + dbl(a[0]) + "))";
        o << " + " << w << " * (t" << ci << "a + t" << ci << "b)";
    }
    o << "; }";
    return o.str();
}

bool is_diag(const PassOp &op) { return op.kind == K_D1 || op.kind == K_D2; }

// The entry of diagonal op `op` (matrix at offset mat) that multiplies
// register k of a stage, as an expression; "" when it is exactly 1.  Bits of
// the op outside the stage select per item.
std::string diag_entry(const Env &e, const PassOp &op, int mat, int k)
{
    const int um = op.hint & 0xf;
    auto en = [&](int idx) { return ((um >> idx) & 1) ? std::string("make_double2(1.0, 0.0)") : ent(mat + idx); };
    auto unit = [&](int idx) { return ((um >> idx) & 1) != 0; };
    if (op.kind == K_D1) {
        if (op.s0 != kFixed) {
            const int idx = (k >> op.s0) & 1;
            return unit(idx) ? "" : ent(mat + idx);
        }
        if (unit(0) && unit(1)) return "";
        return "zsel(" + bit(e, op.l0, op.p0) + ", " + en(0) + ", " + en(1) + ")";
    }
    const bool r0 = op.s0 != kFixed, r1 = op.s1 != kFixed;
    const int c0 = r0 ? (k >> op.s0) & 1 : 0, c1 = r1 ? (k >> op.s1) & 1 : 0;
    if (r0 && r1) return unit(2 * c0 + c1) ? "" : ent(mat + 2 * c0 + c1);
    if (r0) {
        if (unit(2 * c0) && unit(2 * c0 + 1)) return "";
        return "zsel(" + bit(e, op.l1, op.p1) + ", " + en(2 * c0) + ", " + en(2 * c0 + 1) + ")";
    }
    if (r1) {
        if (unit(c1) && unit(2 + c1)) return "";
        return "zsel(" + bit(e, op.l0, op.p0) + ", " + en(c1) + ", " + en(2 + c1) + ")";
    }
    if (unit(0) && unit(1) && unit(2) && unit(3)) return "";
    const std::string b0 = bit(e, op.l0, op.p0), b1 = bit(e, op.l1, op.p1);
    return "zsel(" + b0 + ", zsel(" + b1 + ", " + en(0) + ", " + en(1) + "), zsel(" + b1 + ", " + en(2) + ", " + en(3) +
           "))";
}

// Phase classes.  ZZ-type diagonal ops (a single RZZ or ZZ^t gate each:
// diag(1, w, w, 1) once the left-out global phase is removed) that share
// their parameter expression (opcode, symbol, scale, offset: the same w in a
// row) multiply amplitude i by w^c(i), c(i) the number of the ops whose two
// bits differ in i -- a QAOA layer's 30 edges are one class, c(i) its cut
// size.  A class of at least kCutMin ops of a diagonal run is applied as one
// lookup of w^c in a table of powers (LDS, built once per workgroup) and one
// complex multiply per amplitude; c is summed from the item's bits once per
// item plus, per register, the class's bits in the stage.  The derived rows
// of the parameter shift move one member's parameter: see cut_apply.
constexpr int kCutMin = 3;
struct CutClass {
    std::vector<const PassOp *> ops;
    int rep = 0;  // pass-relative matrix offset of one member (its entry 1 is w)
    int tab = 0;  // offset of its powers w^0 .. w^ops.size() in the table
    int id = 0;   // its index among the pass's classes
};
bool cut_key(const Group &g, const PassOp &op, std::tuple<int, int, double, double> *key)
{
    if (op.kind != K_D2 || (op.hint & 0xf) != 9) return false;
    if (!g.uniform_slots && g.rows.size() > 1) return false;
    const BuildTask *bt = nullptr;
    for (int k = g.fwd_tasks.begin; k < g.fwd_tasks.end && !bt; k++)
        if (g.tasks[k].out == op.mat && g.tasks[k].kind == BT_PRODUCT) bt = &g.tasks[k];
    if (!bt || bt->mem_count != 1 || bt->diag != 1 || bt->dim != 4) return false;
    const Member &mb = g.members[bt->mem_begin];
    const GateDev &gd = g.gates[mb.gate];
    if ((gd.op != OP_RZZ && gd.op != OP_ZZPOW) || mb.form != FORM_FULL || gd.np != 1) return false;
    const int sl = gd.slot0;
    *key = std::make_tuple((int)gd.op, (int)g.slot_sym[sl], g.slot_scale[sl], g.slot_off[sl]);
    return true;
}
// Splits a diagonal run into its phase classes of at least kCutMin ops (in
// order of first appearance) and the ops left over.
void split_run(const Group *g, const std::vector<const PassOp *> &run, std::vector<CutClass> *classes,
               std::vector<const PassOp *> *rest)
{
    std::map<std::tuple<int, int, double, double>, std::vector<const PassOp *>> by;
    std::vector<std::tuple<int, int, double, double>> order;
    std::vector<char> keyed(run.size(), 0);
    for (size_t i = 0; g && i < run.size(); i++) {
        std::tuple<int, int, double, double> k;
        if (!cut_key(*g, *run[i], &k)) continue;
        if (!by.count(k)) order.push_back(k);
        by[k].push_back(run[i]);
        keyed[i] = 1;
    }
    std::set<const PassOp *> taken;
    for (auto &k : order)
        if ((int)by[k].size() >= kCutMin) {
            CutClass c;
            c.ops = by[k];
            classes->push_back(c);
            for (const PassOp *op : c.ops) taken.insert(op);
        }
    for (const PassOp *op : run)
        if (!taken.count(op)) rest->push_back(op);
}
// The phase classes of a forward pass's stages, in emission order, with
// their table offsets; total table entries in *ntab.
std::vector<CutClass> cut_classes(const Group &g, const Pass &ps, int *ntab)
{
    std::vector<CutClass> all;
    *ntab = 0;
    for (const Stage &st : ps.stages) {
        if (st.dense) continue;
        for (int oi = st.op_begin; oi < st.op_end; oi++) {
            if (!is_diag(ps.ops[oi - ps.op_offset])) continue;
            std::vector<const PassOp *> run;
            int oe = oi;
            for (; oe < st.op_end && is_diag(ps.ops[oe - ps.op_offset]); oe++) run.push_back(&ps.ops[oe - ps.op_offset]);
            std::vector<CutClass> cls;
            std::vector<const PassOp *> rest;
            split_run(&g, run, &cls, &rest);
            for (CutClass &c : cls) {
                c.rep = c.ops[0]->mat - ps.mat_begin;
                c.tab = *ntab;
                c.id = (int)all.size();
                *ntab += (int)c.ops.size() + 1;
                all.push_back(c);
            }
            oi = oe - 1;
        }
    }
    return all;
}
// The code applying phase class c on the registers v of stage st.  In the
// derived rows of the parameter shift one member x of a class may hold
// another w_x (its parameter moved): the workgroup's prologue finds it and the
// amplitudes where its bits differ take the factor w_x / w as well.
std::string cut_apply(const Env &e, const CutClass &c, const Stage &st)
{
    const int R = st.r, NR = 1 << R;
    std::ostringstream o;
    o << "{ uint32_t q_ = 0u";
    std::vector<std::pair<int, std::string>> mixed;  // (register bit, item bit expression)
    std::vector<int> stat(NR, 0);
    for (const PassOp *op : c.ops) {
        const bool r0 = op->s0 != kFixed, r1 = op->s1 != kFixed;
        if (!r0 && !r1)
            o << " + (" << bit(e, op->l0, op->p0) << " ^ " << bit(e, op->l1, op->p1) << ")";
        else if (r0 && r1) {
            for (int k = 0; k < NR; k++) stat[k] += ((k >> op->s0) ^ (k >> op->s1)) & 1;
        } else {
            mixed.emplace_back(r0 ? op->s0 : op->s1, r0 ? bit(e, op->l1, op->p1) : bit(e, op->l0, op->p0));
        }
    }
    o << ";";
    for (size_t j = 0; j < mixed.size(); j++) o << " const uint32_t m" << j << "_ = " << mixed[j].second << ";";
    for (int k = 0; k < NR; k++) {
        std::ostringstream cnt;
        int cst = stat[k];
        cnt << "q_";
        for (size_t j = 0; j < mixed.size(); j++) {
            if ((k >> mixed[j].first) & 1) {
                cst += 1;
                cnt << " - m" << j << "_";
            } else {
                cnt << " + m" << j << "_";
            }
        }
        o << " v[" << k << "] = zmul(cutw_[" << c.tab + cst << "u + " << cnt.str() << "], v[" << k << "]);";
    }
    o << " }\n";
    // the moved member (uniform over the workgroup): endpoint s is tile bit s,
    // or with bit 7 set global bit s & 127 of the tile's fixed bits
    o << "        if (cutx_[" << c.id << "] != 0xffffffffu) { const uint32_t x_ = cutx_[" << c.id
      << "], sa_ = x_ & 255u, sb_ = (x_ >> 8) & 255u; const double2 r_ = cutr_[" << c.id << "];";
    for (int k = 0; k < NR; k++) {
        uint32_t roff = 0;
        for (int j = 0; j < R; j++)
            if ((k >> j) & 1) roff |= 1u << st.bits[j];
        o << " { const uint32_t i_ = base | " << roff
          << "u; const uint32_t a_ = (sa_ & 128u) ? ((uint32_t)(fb >> (sa_ & 127u)) & 1u) : ((i_ >> sa_) & 1u);"
             " const uint32_t b_ = (sb_ & 128u) ? ((uint32_t)(fb >> (sb_ & 127u)) & 1u) : ((i_ >> sb_) & 1u);"
             " if (a_ ^ b_) v["
          << k << "] = zmul(r_, v[" << k << "]); }";
    }
    o << " }";
    return o.str();
}

// A run of consecutive diagonal ops of a stage as one diagonal: its entries
// are multiplied together over the register bits the run touches (per item,
// with the out-of-stage bits), then each register of the arrays `arrs` is
// multiplied once.  Returns "" when op by op is no more expensive (complex
// multiplies counted).
// A run of one-qubit diagonal ops on register bits: the diagonal is a tensor
// product over the bits, so its 2^m entries are built by doubling (one
// complex multiply per new entry), with the bits' own entries (the product
// of the ops on each bit) as factors.  "" when op by op is no more expensive.
std::string diag_run_tensor(const Env &e, const std::vector<const PassOp *> &run, int R,
                            const std::vector<std::string> &arrs)
{
    std::vector<int> jb;                       // register bits, ascending
    std::map<int, std::vector<const PassOp *>> on;
    for (const PassOp *op : run) {
        if (op->kind != K_D1 || op->s0 == kFixed) return "";
        on[op->s0].push_back(op);
    }
    for (auto &kv : on) jb.push_back(kv.first);
    const int NR = 1 << R;
    std::ostringstream b;
    int mults = 0, direct = 0, nv = 0;
    auto fresh = [&]() { return "t" + N(nv++) + "_"; };
    // per bit: its entries for bit value 0 and 1 ("" = exactly 1)
    std::vector<std::array<std::string, 2>> eb;
    for (int bit : jb) {
        std::array<std::string, 2> v{"", ""};
        for (int x = 0; x < 2; x++)
            for (const PassOp *op : on[bit]) {
                const std::string en = diag_entry(e, *op, op->mat - e.mbase, x << bit);
                if (en.empty()) continue;
                if (v[x].empty()) {
                    v[x] = en;
                } else {
                    const std::string t = fresh();
                    b << "const double2 " << t << " = zmul(" << v[x] << ", " << en << "); ";
                    v[x] = t;
                    mults++;
                }
            }
        eb.push_back(v);
    }
    for (const PassOp *op : run)
        for (int k = 0; k < NR; k++) direct += !diag_entry(e, *op, op->mat - e.mbase, k).empty();
    // doubling over the bits: entry j of the table (bit i of j: bit jb[i])
    std::vector<std::string> tab(1, "");
    for (size_t i = 0; i < jb.size(); i++) {
        std::vector<std::string> nt(tab.size() * 2);
        for (size_t j = 0; j < tab.size(); j++)
            for (int x = 0; x < 2; x++) {
                const std::string &f = eb[i][x];
                std::string r;
                if (tab[j].empty()) r = f;
                else if (f.empty()) r = tab[j];
                else {
                    r = fresh();
                    b << "const double2 " << r << " = zmul(" << tab[j] << ", " << f << "); ";
                    mults++;
                }
                nt[j | ((size_t)x << i)] = r;
            }
        tab.swap(nt);
    }
    auto proj = [&](int k) {
        int j = 0;
        for (size_t i = 0; i < jb.size(); i++)
            if ((k >> jb[i]) & 1) j |= 1 << i;
        return j;
    };
    std::ostringstream a;
    for (const std::string &v : arrs)
        for (int k = 0; k < NR; k++)
            if (!tab[proj(k)].empty()) {
                a << v << "[" << k << "] = zmul(" << tab[proj(k)] << ", " << v << "[" << k << "]); ";
                mults++;
            }
    if (mults >= direct * (int)arrs.size()) return "";
    return "{ " + b.str() + a.str() + "}";
}

std::string diag_run(const Env &e, const std::vector<const PassOp *> &run, int R, const std::vector<std::string> &arrs)
{
    {
        const std::string t = diag_run_tensor(e, run, R, arrs);
        if (!t.empty()) return t;
    }
    int jm = 0;  // register bits the run touches
    for (const PassOp *op : run) {
        if (op->s0 != kFixed) jm |= 1 << op->s0;
        if (op->kind == K_D2 && op->s1 != kFixed) jm |= 1 << op->s1;
    }
    std::vector<int> jb;
    for (int j = 0; j < R; j++)
        if ((jm >> j) & 1) jb.push_back(j);
    const int NJ = 1 << jb.size(), NR = 1 << R;
    auto rep = [&](int j) {  // a register index with the run's bits set as j says
        int k = 0;
        for (size_t i = 0; i < jb.size(); i++)
            if ((j >> i) & 1) k |= 1 << jb[i];
        return k;
    };
    auto proj = [&](int k) {
        int j = 0;
        for (size_t i = 0; i < jb.size(); i++)
            if ((k >> jb[i]) & 1) j |= 1 << i;
        return j;
    };
    std::vector<bool> one(NJ, true);
    std::ostringstream b;
    int fused = 0, direct = 0;
    for (const PassOp *op : run) {
        const int mat = op->mat - e.mbase;
        for (int k = 0; k < NR; k++) direct += !diag_entry(e, *op, mat, k).empty();
        for (int j = 0; j < NJ; j++) {
            const std::string x = diag_entry(e, *op, mat, rep(j));
            if (x.empty()) continue;
            if (one[j]) {
                b << "d" << j << "_ = " << x << "; ";
                one[j] = false;
            } else {
                b << "d" << j << "_ = zmul(d" << j << "_, " << x << "); ";
                fused++;
            }
        }
    }
    std::ostringstream a;
    for (const std::string &v : arrs)
        for (int k = 0; k < NR; k++)
            if (!one[proj(k)]) {
                a << v << "[" << k << "] = zmul(d" << proj(k) << "_, " << v << "[" << k << "]); ";
                fused++;
            }
    if (fused >= direct * (int)arrs.size()) return "";
    std::ostringstream o;
    o << "{ double2";
    for (int j = 0, first = 1; j < NJ; j++)
        if (!one[j]) {
            o << (first ? " " : ", ") << "d" << j << "_";
            first = 0;
        }
    o << "; " << b.str() << a.str() << "}";
    return o.str();
}

// item loop header of a stage: base index of the item and the swizzled
// LDS offsets of its 2^R registers
void stage_head(std::ostream &o, const Env &e, const Stage &st, std::vector<uint32_t> &off)
{
    const int R = st.r;
    off.assign(1u << R, 0);
    for (uint32_t k = 0; k < (1u << R); k++) {
        uint32_t x = 0;
        for (int j = 0; j < R; j++)
            if ((k >> j) & 1) x |= 1u << st.bits[j];
        off[k] = host_sw(x);  // sw is linear over xor: sw(base | x) = sw(base) ^ sw(x)
    }
    o << "    for (uint32_t item = tid; item < " << (1u << (e.t - R)) << "u; item += " << e.nt << "u) {\n";
    o << "        uint32_t base = item;\n";
    for (int j = 0; j < R; j++) o << "        base = ins0(base, " << (int)st.bits[j] << ");\n";
    o << "        const uint32_t sb = sw(base);\n";
    // an offset of 0 the compiler cannot see through, taken anew per item:
    // matrix reads offset by it stay inside the item loop instead of being
    // hoisted above it, where every matrix of the stage would be live at once
    o << "        int z_ = 0;\n";
    if (e.pin) o << "        asm volatile(\"\" : \"+s\"(z_));\n";
}

// Constant single-qubit ops.  A forward op on one qubit whose member gates
// all have constant parameters, the same in every row, has a matrix known on
// the host (the builder's gate table, gate_table_host); when its diagonal is
// d = M00 = M11, real and positive, it is M = d U with U's diagonal exactly 1
// (sqrt X, sqrt Y and sqrt W without their global phases: U off-diagonal in
// {-i, -1, 1, (-1 -/+ i)/sqrt 2}).  Such an op is written out as U's products
// with every entry that is 0 or +-1 or +-i folded in (entries below 1e-15 of
// the largest taken as 0, within 1e-15 of +-1 as +-1: the rounding of the
// closed forms is removed, not added), and the pass multiplies its registers
// once by the product of the d's at the end of its last stage.
struct ConstM1 {
    double u[8];  // U row major, (re, im)
    double d;     // the factor taken out (1 when none)
};
bool const_m1(const Group &g, const PassOp &op, ConstM1 *out)
{
    if (op.kind != K_M1 || op.ctrl) return false;
    if (!g.uniform_slots && g.rows.size() > 1) return false;
    const BuildTask *bt = nullptr;
    for (int k = g.fwd_tasks.begin; k < g.fwd_tasks.end && !bt; k++)
        if (g.tasks[k].out == op.mat && g.tasks[k].kind == BT_PRODUCT) bt = &g.tasks[k];
    if (!bt || bt->dim != 2 || bt->diag != 0) return false;
    double acc[8] = {1, 0, 0, 0, 0, 0, 1, 0};
    for (int mi = 0; mi < bt->mem_count; mi++) {
        const GateDev &gd = g.gates[g.members[bt->mem_begin + mi].gate];
        double eta[3] = {0, 0, 0};
        for (int j = 0; j < gd.np; j++) {
            if (g.slot_sym[gd.slot0 + j] >= 0) return false;
            eta[j] = g.slot_off[gd.slot0 + j];
        }
        double m[32];
        const double *ex = gd.explicit_ >= 0 ? &g.explicit_mats[32 * (size_t)gd.explicit_] : nullptr;
        if (gate_table_host(gd.op, eta, ex, g.members[bt->mem_begin + mi].form, 0, 0, m) != 2) return false;
        double t[8];
        for (int i = 0; i < 2; i++)
            for (int j = 0; j < 2; j++) {
                double re = 0, im = 0;
                for (int k = 0; k < 2; k++) {
                    const double ar = m[2 * (2 * i + k)], ai = m[2 * (2 * i + k) + 1];
                    const double br = acc[2 * (2 * k + j)], bi = acc[2 * (2 * k + j) + 1];
                    re += ar * br - ai * bi;
                    im += ar * bi + ai * br;
                }
                t[2 * (2 * i + j)] = re;
                t[2 * (2 * i + j) + 1] = im;
            }
        std::copy(t, t + 8, acc);
    }
    double big = 0;
    for (double v : acc) big = std::max(big, std::fabs(v));
    for (double &v : acc)
        if (std::fabs(v) <= 1e-15 * big) v = 0.0;
    out->d = 1.0;
    if (acc[1] == 0.0 && acc[7] == 0.0 && acc[0] == acc[6] && acc[0] >= 0.25) out->d = acc[0];
    for (int i = 0; i < 8; i++) out->u[i] = acc[i] / out->d;
    if (out->d != 1.0) out->u[0] = out->u[6] = 1.0;
    // entries within 1e-15 of +-1 are the unit values they stand for (cos and
    // sin of pi/4 differ in their last bit)
    for (double &v : out->u)
        if (std::fabs(std::fabs(v) - 1.0) <= 1e-15) v = v > 0 ? 1.0 : -1.0;
    return true;
}

// One component of c0 x + c1 y (c complex literals, x y register names):
// re: sum c.x w.x - c.y w.y, im: sum c.x w.y + c.y w.x, with zero terms left
// out and unit factors as additions.
std::string cterm_sum(const std::vector<std::pair<const double *, std::string>> &terms, bool im)
{
    std::vector<std::pair<double, std::string>> t;  // coefficient, operand
    for (auto &tm : terms) {
        const double cx = tm.first[0], cy = tm.first[1];
        const std::string &w = tm.second;
        if (!im) {
            if (cx != 0) t.emplace_back(cx, w + ".x");
            if (cy != 0) t.emplace_back(-cy, w + ".y");
        } else {
            if (cx != 0) t.emplace_back(cx, w + ".y");
            if (cy != 0) t.emplace_back(cy, w + ".x");
        }
    }
    if (t.empty()) return "0.0";
    // unit terms first (additions), then the others as an fma chain on them
    std::stable_sort(t.begin(), t.end(), [](const std::pair<double, std::string> &a, const std::pair<double, std::string> &b) {
        return (std::fabs(a.first) == 1.0) > (std::fabs(b.first) == 1.0);
    });
    std::string acc;
    for (auto &tm : t) {
        const double c = tm.first;
        if (acc.empty()) {
            acc = c == 1.0 ? tm.second : c == -1.0 ? "(-" + tm.second + ")" : "(" + dbl(c) + " * " + tm.second + ")";
        } else if (c == 1.0) {
            acc = "(" + acc + " + " + tm.second + ")";
        } else if (c == -1.0) {
            acc = "(" + acc + " - " + tm.second + ")";
        } else {
            acc = "fma(" + dbl(c) + ", " + tm.second + ", " + acc + ")";
        }
    }
    return acc;
}

std::string const_m1_code(const ConstM1 &cm, const PassOp &op, int R)
{
    std::ostringstream o;
    const int J = op.s0;
    for (int k = 0; k < (1 << R); k++) {
        if ((k >> J) & 1) continue;
        const int kk = k | (1 << J);
        o << "{ const double2 x_ = v[" << k << "], y_ = v[" << kk << "]; ";
        o << "v[" << k << "] = make_double2(" << cterm_sum({{cm.u + 0, "x_"}, {cm.u + 2, "y_"}}, false) << ", "
          << cterm_sum({{cm.u + 0, "x_"}, {cm.u + 2, "y_"}}, true) << "); ";
        o << "v[" << kk << "] = make_double2(" << cterm_sum({{cm.u + 4, "x_"}, {cm.u + 6, "y_"}}, false) << ", "
          << cterm_sum({{cm.u + 4, "x_"}, {cm.u + 6, "y_"}}, true) << "); } ";
    }
    return o.str();
}

// A forward stage on the tile lp.  scale: the factor the pass's constant ops
// left out, multiplied into the registers at the end of the stage ("" = none).
void forward_stage(std::ostream &o, const Env &e, const Pass &ps, const Stage &st, const std::string &scale = "")
{
    const int R = st.r, NR = 1 << R;
    std::vector<uint32_t> off;
    o << "    {\n";
    stage_head(o, e, st, off);
    o << "        double2 v[" << NR << "];\n";
    for (int k = 0; k < NR; k++) o << "        v[" << k << "] = up2(lp[sb ^ " << off[k] << "u]);\n";
    if (st.dense) {
        o << "        rdense<" << R << ">(v, " << e.G << " + (z_ + " << st.mat << "));\n";
    } else {
        for (int oi = st.op_begin; oi < st.op_end; oi++) {
            const PassOp &op = ps.ops[oi - ps.op_offset];
            if (is_diag(op)) {
                std::vector<const PassOp *> run;
                int oe = oi;
                for (; oe < st.op_end && is_diag(ps.ops[oe - ps.op_offset]); oe++)
                    run.push_back(&ps.ops[oe - ps.op_offset]);
                if (e.cuts) {
                    // phase classes first (diagonal ops commute), then the rest
                    std::vector<CutClass> cls;
                    std::vector<const PassOp *> rest;
                    split_run(e.fgrp, run, &cls, &rest);
                    if (!cls.empty()) {
                        for (size_t ci = 0; ci < cls.size(); ci++)
                            o << "        " << cut_apply(e, (*e.cuts)[e.cut_next++], st) << "\n";
                        const std::string c = rest.size() > 1 ? diag_run(e, rest, R, {"v"}) : "";
                        if (!c.empty())
                            o << "        " << c << "\n";
                        else
                            for (const PassOp *ro : rest) o << "        " << apply(e, *ro, R, ro->mat - e.mbase, "v") << "\n";
                        oi = oe - 1;
                        continue;
                    }
                }
                const std::string c = run.size() > 1 ? diag_run(e, run, R, {"v"}) : "";
                if (!c.empty()) {
                    o << "        " << c << "\n";
                    oi = oe - 1;
                    continue;
                }
            }
            ConstM1 cm;
            if (e.fgrp && const_m1(*e.fgrp, op, &cm)) {
                o << "        " << const_m1_code(cm, op, R) << "\n";
                continue;
            }
            o << "        " << apply(e, op, R, op.mat - e.mbase, "v") << "\n";
        }
    }
    if (!scale.empty())
        for (int k = 0; k < NR; k++) o << "        v[" << k << "].x *= " << scale << "; v[" << k << "].y *= " << scale << ";\n";
    for (int k = 0; k < NR; k++) o << "        lp[sb ^ " << off[k] << "u] = down2(v[" << k << "]);\n";
    o << "    }\n    }\n    __syncthreads();\n";
}

// The product of the factors the constant ops of a pass's stages leave out
// ("" when it is 1), written in where the last stage applies it.
std::string pass_scale(const Env &e, const Pass &ps)
{
    if (!e.fgrp) return "";
    double s = 1.0;
    for (const Stage &st : ps.stages) {
        if (st.dense) continue;
        for (int oi = st.op_begin; oi < st.op_end; oi++) {
            ConstM1 cm;
            if (const_m1(*e.fgrp, ps.ops[oi - ps.op_offset], &cm)) s *= cm.d;
        }
    }
    return s == 1.0 ? "" : dbl(s);
}

// A reverse stage on the tiles lp (psi) and lf (phi); the gradient partials
// of its parameters stay in registers over the items, then one wavefront
// sum each goes to the wave's accumulator row.
void reverse_stage(std::ostream &o, const Env &e, const Pass &ps, const Stage &st)
{
    const int R = st.r, NR = 1 << R;
    std::vector<uint32_t> off;
    std::vector<std::pair<int, int>> grads;  // (register, gradient slot)
    for (int oi = st.op_begin; oi < st.op_end; oi++) {
        const PassOp &op = ps.ops[oi - ps.op_offset];
        for (int j = 0; j < op.ngrad; j++) grads.emplace_back((int)grads.size(), op.gslot[j]);
    }
    o << "    {\n";
    if (!grads.empty()) o << "    double g[" << grads.size() << "] = {};\n";
    stage_head(o, e, st, off);
    o << "        double2 v[" << NR << "], f[" << NR << "];\n";
    for (int k = 0; k < NR; k++)
        o << "        v[" << k << "] = up2(lp[sb ^ " << off[k] << "u]); f[" << k << "] = up2(lf[sb ^ " << off[k]
          << "u]);\n";
    int gk = 0;
    for (int oi = st.op_begin; oi < st.op_end; oi++) {
        const PassOp &op = ps.ops[oi - ps.op_offset];
        // A run of diagonal ops whose gradients all come from diagonal
        // generators: the ops commute with each other and with the
        // generators, so Im<f|G|v> is the same before every op of the run;
        // all its gradients are taken first, then the run is applied to v
        // and f as one diagonal.
        if (is_diag(op) && e.grp) {
            std::vector<const PassOp *> run;
            std::vector<std::string> dots;
            int gkr = gk;
            for (int oe = oi; oe < st.op_end && is_diag(ps.ops[oe - ps.op_offset]); oe++) {
                const PassOp &ro = ps.ops[oe - ps.op_offset];
                std::vector<std::string> od;
                bool ok = true;
                for (int j = 0; j < ro.ngrad && ok; j++) {
                    std::vector<GenTerm> gt;
                    ok = op_generator(*e.grp, ro, j, &gt);
                    for (const GenTerm &tm : gt) ok = ok && tm.x == 0;
                    const std::string c = ok ? gen_dot(e, ro, R, gt, "g[" + N(gkr + j) + "]") : "";
                    ok = ok && !c.empty();
                    od.push_back(c);
                }
                if (!ok) break;
                run.push_back(&ro);
                dots.insert(dots.end(), od.begin(), od.end());
                gkr += ro.ngrad;
            }
            const std::string c = run.size() > 1 ? diag_run(e, run, R, {"v", "f"}) : "";
            if (!c.empty()) {
                for (const std::string &d : dots) o << "        " << d << "\n";
                o << "        " << c << "\n";
                if (e.pin) o << "        __builtin_amdgcn_sched_barrier(0);\n";
                gk = gkr;
                oi = oi + (int)run.size() - 1;
                continue;
            }
        }
        // gradients from the gate's generator on the registers before the op
        // (no derivative matrix read), else Re(conj(f) dW v) after W^dagger v
        std::vector<std::string> gd;
        for (int j = 0; j < op.ngrad && e.grp; j++) {
            std::vector<GenTerm> gt;
            const std::string c = op_generator(*e.grp, op, j, &gt) ? gen_dot(e, op, R, gt, "g[" + N(gk + j) + "]") : "";
            if (c.empty()) break;
            gd.push_back(c);
        }
        if ((int)gd.size() == op.ngrad) {
            for (const std::string &c : gd) o << "        " << c << "\n";
            gk += op.ngrad;
            o << "        " << apply(e, op, R, op.mat - e.mbase, "v") << "\n";
        } else {
            o << "        " << apply(e, op, R, op.mat - e.mbase, "v") << "\n";
            for (int j = 0; j < op.ngrad; j++)
                o << "        g[" << gk++ << "] += " << dot(e, op, R, op.dmat[j] - e.mbase) << ";\n";
        }
        o << "        " << apply(e, op, R, op.mat - e.mbase, "f") << "\n";
        // keep each op's matrix reads next to the op: scheduled ahead they
        // would hold every matrix of the stage in registers at once
        if (e.pin) o << "        __builtin_amdgcn_sched_barrier(0);\n";
    }
    for (int k = 0; k < NR; k++)
        o << "        lp[sb ^ " << off[k] << "u] = down2(v[" << k << "]); lf[sb ^ " << off[k] << "u] = down2(f[" << k
          << "]);\n";
    o << "    }\n";
    for (auto &gs : grads) {
        if (e.gacc_reg)
            o << "    gacc_[" << gs.second + e.gshift << "] += g[" << gs.first << "];\n";
        else
            o << "    { const double s_ = wave_sum(g[" << gs.first << "]); if ((tid & 63) == 0) acc[(tid >> 6) * "
              << e.acc_stride << " + " << gs.second << " + " << e.acc_shift << "] += s_; }\n";
    }
    o << "    }\n    __syncthreads();\n";
}

// Gradient slots of a reverse tile pass that keep per-thread register sums
// over the workgroup's tiles (two VGPRs each).
constexpr int kRevRegGrads = 32;
// With kRevPrefetch the reverse tile passes load the next tile's psi and phi
// into registers while the current tile's stages run, as the forward passes
// do.  Off: the 64 VGPRs it takes leave no room for the register gradient
// sums, and either way it measured slower (VQE reverse passes 47.5-48.5 ms
// per step with it, 45.7 ms without it and with the register sums).
constexpr bool kRevPrefetch = false;

const char kHead[] =
    "namespace tq {\n"
    "__device__ __forceinline__ double2 zsel(uint32_t c, double2 a, double2 b) { return c ? b : a; }\n"
    "__device__ __forceinline__ bool zeq(double2 a, double2 b) { return a.x == b.x && a.y == b.y; }\n"
    "__device__ __forceinline__ double2 zpow(double2 w, uint32_t n)\n"
    "{ double2 r = make_double2(1.0, 0.0); while (n) { if (n & 1u) r = zmul(r, w); w = zmul(w, w); n >>= 1; } return r; }\n";

} // namespace

int resident_threads(const Group &g)
{
    // one thread per item of a three-bit stage when the reverse stages are
    // that wide (measured fastest on 10 qubits: 128 threads 0.144 ms, 256
    // threads 0.152 ms, against 0.152 ms for 256 threads and two-bit reverse
    // stages), else four wavefronts
    bool wide = false;
    for (const Pass &ps : g.rev)
        for (const Stage &st : ps.stages) wide |= st.r > kStageBitsRevResident;
    if (!wide) return kThreads;
    return std::min(kThreads, std::max(64, 1 << std::max(g.n - kStageBitsRev, 0)));
}

std::string resident_source(const Group &g)
{
    std::ostringstream o;
    const int n = g.n, nt = resident_threads(g);
    o << kHead
      << "extern \"C\" __global__ __launch_bounds__(" << nt << ") void tq_resident_spec(ResArgs a)\n{\n"
         "    extern __shared__ __align__(16) unsigned char smem[];\n"
         "    double *acc = reinterpret_cast<double *>(smem);\n"
         "    float2 *lp = reinterpret_cast<float2 *>(acc + 4 * a.nacc);\n"
         "    float2 *lf = lp + "
      << (1u << n)
      << "u;\n"
         "    const SMat M = smat(a.mats + (int64_t)blockIdx.x * a.mat_stride);\n"
         "    const int tid = threadIdx.x;\n"
         "    resident_begin(a, M, acc, lp, tid, " << nt << ");\n";
    Env e{n, 0, "M", false, "a.nacc", "a.gacc"};
    e.pin = false;  // two waves per SIMD: registers to spare, latency to hide
    e.nt = nt;
    e.grp = &g;
    e.fgrp = &g;
    for (const Pass &ps : g.fwd) {
        const std::string scale = pass_scale(e, ps);
        for (size_t si = 0; si < ps.stages.size(); si++)
            forward_stage(o, e, ps, ps.stages[si], si + 1 == ps.stages.size() ? scale : "");
    }
    o << "    resident_middle(a, acc, lp, lf, blockIdx.x, tid, " << nt << ");\n"
         "    if (a.grad) {\n";
    for (const Pass &ps : g.rev)
        for (const Stage &st : ps.stages) reverse_stage(o, e, ps, st);
    o << "    }\n"
         "    resident_end(a, acc, blockIdx.x, tid, " << nt << ");\n"
         "}\n"
         "} // namespace tq\n";
    return o.str();
}

namespace {

// Tile loads and stores of a generated forward pass with the tile's geometry
// written in (every pass but the first, which generates the product state):
// thread tid holds the pairs l = 2 tid + 512 k (k < 2^t / 512) of the tile.
// The global offset of l is a per-thread part -- the tid bits deposited at
// their global positions -- plus a constant per k, and its LDS position sw(l)
// is one of two per-thread values (by the parity of k) plus 512 k, an
// immediate offset: no table lookups and no guards, all loads of a tile
// issued back to back.
bool direct_io(const Pass &ps) { return !ps.product_init && ps.geom.t >= 9 && ps.geom.c >= 1; }

// global index bit of tile-local bit b
int gpos(const TileGeom &gm, int b) { return b < gm.c ? b : gm.hb[b - gm.c]; }

// With kFwdPrefetch the next tile's loads are issued right after the current
// tile is in LDS, into registers held over its stages, so that every
// workgroup streams its next tile while it computes; the registers this takes
// leave three workgroups per CU instead of four.
constexpr bool kFwdPrefetch = true;

void direct_io_setup(std::ostream &o, const TileGeom &gm)
{
    o << "    const uint32_t tb_ = (uint32_t)tid << 1;\n"
         "    const uint32_t la0_ = tb_ ^ ((tb_ >> 5) & 15u), la1_ = la0_ ^ 16u, lb0_ = la0_ ^ 1u, lb1_ = la1_ ^ 1u;\n"
         "    uint64_t toff_ = 0;\n";
    for (int j = 0; j < 8; j++)
        o << "    toff_ |= (uint64_t)(((uint32_t)tid >> " << j << ") & 1u) << " << gpos(gm, j + 1) << ";\n";
}

uint64_t chunk_offset(const TileGeom &gm, int k)
{
    uint64_t o = 0;
    for (int m = 0; 9 + m < gm.t; m++)
        if ((k >> m) & 1) o |= 1ull << gpos(gm, 9 + m);
    return o;
}

void direct_load(std::ostream &o, const TileGeom &gm, const std::string &fb, const std::string &dst,
                 const std::string &row = "c.st")
{
    const int K = 1 << (gm.t - 9);
    o << "    { const float2 *src_ = " << row << " + (" << fb << " | toff_);\n";
    for (int k = 0; k < K; k++)
        o << "      " << dst << "[" << k << "] = *reinterpret_cast<const float4 *>(src_ + " << chunk_offset(gm, k)
          << "ull);\n";
    o << "    }\n";
}

void direct_to_lds(std::ostream &o, const TileGeom &gm, const std::string &srcv, const std::string &lds = "lp")
{
    const int K = 1 << (gm.t - 9);
    for (int k = 0; k < K; k++) {
        const std::string p = (k & 1) ? "1_" : "0_";
        o << "    " << lds << "[la" << p << " + " << 512 * k << "u] = make_float2(" << srcv << "[" << k << "].x, " << srcv << "[" << k
          << "].y); " << lds << "[lb" << p << " + " << 512 * k << "u] = make_float2(" << srcv << "[" << k << "].z, " << srcv << "["
          << k << "].w);\n";
    }
}

void direct_store(std::ostream &o, const TileGeom &gm, const std::string &fb, const std::string &row = "c.st",
                  const std::string &lds = "lp")
{
    const int K = 1 << (gm.t - 9);
    o << "    { float2 *dst_ = " << row << " + (" << fb << " | toff_);\n";
    for (int k = 0; k < K; k++) {
        const std::string p = (k & 1) ? "1_" : "0_";
        o << "      { const float2 u0 = " << lds << "[la" << p << " + " << 512 * k << "u], u1 = " << lds << "[lb" << p
          << " + " << 512 * k
          << "u]; *reinterpret_cast<float4 *>(dst_ + " << chunk_offset(gm, k)
          << "ull) = make_float4(u0.x, u0.y, u1.x, u1.y); }\n";
    }
    o << "    }\n";
}

} // namespace

std::string pass_kernel_source(const Group &g, int pass)
{
    std::ostringstream o;
    const Pass &ps = g.fwd[pass];
    const TileGeom &gm = ps.geom;
    const bool dio = direct_io(ps), pre = dio && kFwdPrefetch;
    const int64_t NT = 1ll << (gm.n - gm.t);
    // at most 128 registers (four workgroups of the tile's LDS share a CU), or
    // 168 with the prefetch registers (three); a pass with four-bit stages
    // (16 amplitudes and up to 16 diagonal entries per thread) may take 256,
    // so that it never spills -- the waves per SIMD follow what it uses
    int maxr = 0;
    for (const Stage &st : ps.stages) maxr = std::max(maxr, (int)st.r);
    const int minwg = maxr >= 4 ? 2 : pre ? 3 : 4;
    o << "extern \"C\" __global__ __launch_bounds__(256, " << minwg << ") void tq_fwd_" << pass
      << "(PassArgs a)\n{\n"
         "    extern __shared__ __align__(16) unsigned char smem[];\n"
         "    const PassCtx c = pass_setup(a, smem);\n"
         // op matrices through the scalar cache (SGPR operands of the FMAs),
         // not from the LDS copy: the stages' LDS traffic is the tile alone
         "    const SMat M = smat(a.mats + (int64_t)c.row * a.mat_stride + a.mat_begin);\n"
         "    const SMat G = smat(a.mats + (int64_t)c.row * a.mat_stride);\n"
         "    float2 *lp = c.lds;\n"
         "    const int tid = threadIdx.x;\n";
    Env e{gm.t, ps.mat_begin, "G", gm.fixed_mask != 0, "", ""};
    e.fgrp = &g;
    int ntab = 0;
    const std::vector<CutClass> cuts = cut_classes(g, ps, &ntab);
    if (!cuts.empty()) {
        // per phase class, once per workgroup: the w most members hold (the
        // first three include two equal ones), the member that differs if
        // any (a derived row's moved parameter; at most one per class: a move
        // changes one parameter slot) with w_x / w, and the powers of w
        e.cuts = &cuts;
        const size_t nc = cuts.size();
        o << "    __shared__ double2 cutw_[" << ntab << "], cutm_[" << nc << "], cutr_[" << nc << "];\n"
          << "    __shared__ uint32_t cutx_[" << nc << "];\n"
          << "    if (tid == 0) {\n";
        auto endpoint = [](uint8_t l, uint8_t p) { return l != kFixed ? (uint32_t)l : (0x80u | p); };
        for (const CutClass &c : cuts) {
            const int b = ps.mat_begin;
            o << "    { const double2 w0_ = M[" << c.ops[0]->mat - b << " + 1], w1_ = M[" << c.ops[1]->mat - b
              << " + 1], w2_ = M[" << c.ops[2]->mat - b << " + 1];\n"
              << "      const double2 wm_ = (zeq(w0_, w1_) || zeq(w0_, w2_)) ? w0_ : w1_;\n"
              << "      uint32_t x_ = 0xffffffffu; double2 r_ = make_double2(1.0, 0.0);\n";
            for (const PassOp *op : c.ops)
                o << "      { const double2 u_ = M[" << op->mat - b << " + 1]; if (!zeq(u_, wm_)) { x_ = "
                  << (endpoint(op->l0, op->p0) | (endpoint(op->l1, op->p1) << 8))
                  << "u; r_ = zmul(u_, make_double2(wm_.x, -wm_.y)); } }\n";
            o << "      cutm_[" << c.id << "] = wm_; cutr_[" << c.id << "] = r_; cutx_[" << c.id << "] = x_; }\n";
        }
        o << "    }\n    __syncthreads();\n";
        for (const CutClass &c : cuts)
            o << "    for (int j_ = tid; j_ <= " << c.ops.size() << "; j_ += 256) cutw_[" << c.tab << " + j_] = zpow(cutm_["
              << c.id << "], (uint32_t)j_);\n";
        o << "    __syncthreads();\n";
    }
    const std::string scale = pass_scale(e, ps);
    auto stages = [&]() {
        for (size_t si = 0; si < ps.stages.size(); si++)
            forward_stage(o, e, ps, ps.stages[si], si + 1 == ps.stages.size() ? scale : "");
    };
    if (!dio) {
        o << "    for (int64_t tile = c.w; tile < " << NT << "ll; tile += a.wg_per_row) {\n"
          << "    const uint64_t fb = pdep64((uint64_t)tile, " << gm.fixed_mask << "ull);\n"
             "    pass_load(a, c, fb);\n"
             "    __syncthreads();\n";
        stages();
        o << "    pass_store(a, c, fb);\n"
             "    __syncthreads();\n"
             "    }\n"
             "}\n";
        return o.str();
    }
    direct_io_setup(o, gm);
    const int K = 1 << (gm.t - 9);
    o << "    float4 nx_[" << K << "];\n";
    if (pre) {
        o << "    if (c.w < " << NT << "ll) {\n";
        direct_load(o, gm, "pdep64((uint64_t)c.w, " + std::to_string(gm.fixed_mask) + "ull)", "nx_");
        o << "    }\n";
    }
    o << "    for (int64_t tile = c.w; tile < " << NT << "ll; tile += a.wg_per_row) {\n"
      << "    const uint64_t fb = pdep64((uint64_t)tile, " << gm.fixed_mask << "ull);\n";
    if (!pre) direct_load(o, gm, "fb", "nx_");
    direct_to_lds(o, gm, "nx_");
    o << "    __syncthreads();\n";
    if (pre) {
        // the next tile's loads, in flight during this tile's stages
        o << "    if (tile + a.wg_per_row < " << NT << "ll) {\n"
          << "    const uint64_t fbn_ = pdep64((uint64_t)(tile + a.wg_per_row), " << gm.fixed_mask << "ull);\n";
        direct_load(o, gm, "fbn_", "nx_");
        o << "    }\n";
    }
    stages();
    direct_store(o, gm, "fb");
    o << "    __syncthreads();\n"
         "    }\n"
         "}\n";
    return o.str();
}

std::string rev_pass_kernel_source(const Group &g, int pass)
{
    std::ostringstream o;
    int gbase = 0;
    for (int pi = 0; pi < pass; pi++)
        for (const PassOp &op : g.rev[pi].ops) gbase += op.ngrad;
    const Pass &ps = g.rev[pass];
    const TileGeom &gm = ps.geom;
    int gcount = 0;
    for (const PassOp &op : ps.ops) gcount += op.ngrad;
    const bool dio = gm.t >= 9 && gm.c >= 1;
    o << "extern \"C\" __global__ __launch_bounds__(256, 2) void tq_rev_" << pass
      << "(RevArgs a)\n{\n"
         "    extern __shared__ __align__(16) unsigned char smem[];\n"
         "    const RevCtx c = rev_setup(a, smem);\n"
         // matrices through the scalar cache, as in the forward passes
         "    const SMat M = smat(a.mats + (int64_t)c.row * a.mat_stride + a.mat_begin);\n"
         "    float2 *lp = c.lp, *lf = c.lf;\n"
         "    double *acc = c.acc;\n"
         "    const int tid = threadIdx.x;\n";
    if (dio) direct_io_setup(o, gm);
    const bool greg = gcount > 0 && gcount <= kRevRegGrads;
    if (greg) o << "    double gacc_[" << gcount << "] = {};\n";
    const long long NT = 1ll << (gm.n - gm.t);
    const int K = dio ? 1 << (gm.t - 9) : 0;
    const bool pre = dio && kRevPrefetch;
    if (pre) {
        o << "    float4 xp_[" << K << "], xf_[" << K << "];\n"
          << "    if (c.w < " << NT << "ll) {\n";
        const std::string f0 = "pdep64((uint64_t)c.w, " + std::to_string(gm.fixed_mask) + "ull)";
        direct_load(o, gm, f0, "xp_", "c.sp");
        direct_load(o, gm, f0, "xf_", "c.sf");
        o << "    }\n";
    }
    o << "    for (int64_t tile = c.w; tile < " << NT << "ll; tile += a.wg_per_row) {\n"
      << "    const uint64_t fb = pdep64((uint64_t)tile, " << gm.fixed_mask << "ull);\n";
    if (pre) {
        direct_to_lds(o, gm, "xp_", "lp");
        direct_to_lds(o, gm, "xf_", "lf");
        o << "    __syncthreads();\n";
        // the next tile's loads, in flight during this tile's stages
        o << "    if (tile + a.wg_per_row < " << NT << "ll) {\n"
          << "    const uint64_t fbn_ = pdep64((uint64_t)(tile + a.wg_per_row), " << gm.fixed_mask << "ull);\n";
        direct_load(o, gm, "fbn_", "xp_", "c.sp");
        direct_load(o, gm, "fbn_", "xf_", "c.sf");
        o << "    }\n";
    } else if (dio) {
        o << "    { float4 xp_[" << K << "], xf_[" << K << "];\n";
        direct_load(o, gm, "fb", "xp_", "c.sp");
        direct_load(o, gm, "fb", "xf_", "c.sf");
        direct_to_lds(o, gm, "xp_", "lp");
        direct_to_lds(o, gm, "xf_", "lf");
        o << "    }\n    __syncthreads();\n";
    } else {
        o << "    rev_load(a, c, fb);\n    __syncthreads();\n";
    }
    // accumulator rows of gcount slots, the pass's first slot at column 0
    Env e{gm.t, ps.mat_begin, "G", gm.fixed_mask != 0, N(gcount), N(-gbase)};
    e.grp = &g;
    e.gacc_reg = greg;
    e.gshift = -gbase;
    for (const Stage &st : ps.stages) reverse_stage(o, e, ps, st);
    if (dio) {
        o << "    if (a.store) {\n";
        direct_store(o, gm, "fb", "c.sp", "lp");
        direct_store(o, gm, "fb", "c.sf", "lf");
        o << "    }\n";
    } else {
        o << "    rev_store(a, c, fb);\n";
    }
    o << "    __syncthreads();\n"
         "    }\n";
    if (greg) {
        for (int i = 0; i < gcount; i++)
            o << "    { const double s_ = wave_sum(gacc_[" << i << "]); if ((tid & 63) == 0) acc[(tid >> 6) * " << gcount
              << " + " << i << "] += s_; }\n";
        o << "    __syncthreads();\n";
    }
    o << "    rev_finish(a, c);\n"
         "}\n";
    return o.str();
}

namespace {

// Partner reads la[b ^ host_sw(NT q)] with b < NT a swizzled thread index:
// the swizzle only moves bits below NT, so the xor splits into b ^ low (a
// base pointer per distinct low part) plus a multiple of NT that the LDS read
// takes as an immediate offset.
struct LdsSplit {
    uint32_t low, high;
};
LdsSplit lds_split(uint32_t NT, uint32_t q)
{
    const uint32_t v = host_sw(NT * q);
    return LdsSplit{v & (NT - 1), v & ~(NT - 1)};
}

// A mask in global index bits as tile-local bits of geometry gm.
uint32_t local_mask(const TileGeom &gm, uint64_t m)
{
    uint32_t v = 0;
    for (int k = 0; k < gm.c; k++)
        if ((m >> k) & 1) v |= 1u << k;
    for (int k = 0; k < gm.h; k++)
        if ((m >> gm.hb[k]) & 1) v |= 1u << (gm.c + k);
    return v;
}

} // namespace

namespace {

// phi = g H psi over the tile of one pass: per thread 16 amplitudes (the top
// four bits of the tile index) in four chunks of four; per chunk and term
// group (same X mask on the tile) one partner read per amplitude, per term
// two FMAs with the term's coefficient c' = coeff i^ny chi_z(x) signed by
// chi_z of the output amplitude (fixed and thread bits: once per group and
// chunk, register bits: at compile time).
void hphi_pass(std::ostream &o, const PauliPass &pp, int pi)
{
    const TileGeom &gm = pp.geom;
    const int t = gm.t, P = 16, RC = 4, tb = t - 4, NT = 1 << tb, NW = NT / 64;
    struct TT {
        uint32_t zlo, zhi;
        uint64_t zF;
        double C;  // c' = C (real) or i C (imaginary)
        bool im;
    };
    std::map<uint32_t, std::vector<TT>> groups;
    for (const SpecTerm &tm : pp.terms) {
        const uint32_t xT = local_mask(gm, tm.x), zT = local_mask(gm, tm.z);
        const int ny = tm.ny & 3;
        const double chi = (__builtin_popcountll(tm.x & tm.z) & 1) ? -1.0 : 1.0;
        const double C = tm.coeff * chi * (ny >= 2 ? -1.0 : 1.0);
        groups[xT].push_back(TT{zT & (uint32_t)(NT - 1), zT >> tb, tm.z & gm.fixed_mask, C, (ny & 1) != 0});
    }
    o << "extern \"C\" __global__ __launch_bounds__(" << NT << ") void tq_hphi_" << pi
      << "(HPhiArgs a)\n{\n"
         "    extern __shared__ __align__(16) unsigned char smem[];\n"
         "    float2 *la = reinterpret_cast<float2 *>(smem);\n"
         "    uint64_t *hi_off = reinterpret_cast<uint64_t *>(la + "
      << (1 << t)
      << ");\n"
         "    double *red = reinterpret_cast<double *>(hi_off + "
      << (1 << gm.h)
      << ");\n"
         "    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;\n"
         "    const int row = blockIdx.x / a.wg_per_row, w = blockIdx.x % a.wg_per_row;\n"
         "    const int64_t ro = (int64_t)cget(a.rows, row) * a.row_stride;\n"
         "    float2 *ps = const_cast<float2 *>(a.psi) + ro;\n"
         "    float2 *pf = a.phi + ro;\n"
         "    const double gw = (double)a.upstream[(int64_t)cget(a.brows, row) * a.K];\n"
         "    build_hi_off(a.g, hi_off);\n"
         "    __syncthreads();\n"
         "    const TileCtx tc{hi_off, "
      << ((1u << gm.c) - 1) << "u, " << gm.c
      << "};\n"
         "    const uint32_t st = sw((uint32_t)tid);\n"
         "    uint32_t tz = (uint32_t)tid;\n"
         "    double e = 0.0;\n"
         "    for (int64_t tile = w; tile < "
      << (1ll << (gm.n - t)) << "ll; tile += a.wg_per_row) {\n"
      << "    const uint64_t fb = pdep64((uint64_t)tile, " << gm.fixed_mask << "ull);\n"
      << "    tile_copy<true>(tc, la, ps, fb, " << (1 << t) << ");\n"
      << "    __syncthreads();\n";
    std::vector<std::pair<uint32_t, const std::vector<TT> *>> gl;
    for (auto &g : groups) gl.emplace_back(g.first, &g.second);
    for (int ch = 0; ch < P / RC; ch++) {
        // the thread index made opaque anew per chunk: what is derived from
        // it (partner offsets, signed coefficients) is recomputed next to its
        // use instead of being held across chunks and tiles
        // zc: a zero the compiler cannot see through, xored into each
        // coefficient's words so that they are formed next to their use
        // (hoisted out of the tile loop, hundreds of them would be held in
        // registers and spilled)
        o << "    {\n    asm volatile(\"\" : \"+v\"(tz));\n"
          << "    uint32_t zc = 0u;\n    asm volatile(\"\" : \"+v\"(zc));\n"
          // thread bits and the tile number side by side: a term's sign is
          // the parity of one masked word
          << "    const uint32_t vz = tz | ((uint32_t)tile << " << tb << ");\n"
          << "    double2 acc[" << RC << "];\n"
          << "#pragma unroll\n    for (int r = 0; r < " << RC << "; r++) acc[r] = make_double2(0.0, 0.0);\n";
        for (size_t gi = 0; gi < gl.size(); gi++) {
            const uint32_t xT = gl[gi].first, xhi = xT >> tb;
            const std::vector<TT> &tts = *gl[gi].second;
            o << "    {\n";
            o << "        const uint32_t pt = sw(tz ^ " << (xT & (uint32_t)(NT - 1)) << "u);\n";
            std::set<uint32_t> lows;
            for (int rr = 0; rr < RC; rr++) lows.insert(lds_split(NT, (ch * RC + rr) ^ xhi).low);
            for (uint32_t L : lows) o << "        const float2 *lp" << L << " = la + (pt ^ " << L << "u);\n";
            for (size_t j = 0; j < tts.size(); j++) {
                const TT &tt = tts[j];
                // the sign flips the coefficient's sign bit (integer ops: no
                // per-term lane masks held in scalar registers)
                uint64_t zt = 0;  // the term's Z bits among the fixed bits, as tile-number bits
                for (int b = 0, k = 0; b < gm.n; b++)
                    if ((gm.fixed_mask >> b) & 1) zt |= ((tt.zF >> b) & 1ull) << k++;
                const uint64_t m = (uint64_t)tt.zlo | (zt << tb);
                uint64_t cb;
                std::memcpy(&cb, &tt.C, sizeof cb);
                const uint32_t chi = (uint32_t)(cb >> 32), clo = (uint32_t)cb;
                o << "        const double k" << j << " = __hiloint2double((int)(" << chi << "u ^ ";
                if (!m) o << "zc";
                else o << "((uint32_t)(__popc(vz & " << m << "u) & 1) << 31)";
                o << "), (int)(" << clo << "u ^ zc));\n";
            }
            for (int rr = 0; rr < RC; rr++) {
                const int r = ch * RC + rr;
                const LdsSplit pw = lds_split(NT, r ^ xhi);
                o << "        { const double2 p = up2(lp" << pw.low << "[" << pw.high << "]);";
                for (size_t j = 0; j < tts.size(); j++) {
                    const TT &tt = tts[j];
                    const bool neg = __builtin_popcount(tt.zhi & (uint32_t)r) & 1;
                    const std::string k = (neg ? "-k" : "k") + N((long)j);
                    const std::string A = "acc[" + N(rr) + "]";
                    if (!tt.im)
                        o << " " << A << ".x = fma(" << k << ", p.x, " << A << ".x); " << A << ".y = fma(" << k << ", p.y, "
                          << A << ".y);";
                    else  // i k p = k (-p.y, p.x)
                        o << " " << A << ".x = fma(" << k << ", -p.y, " << A << ".x); " << A << ".y = fma(" << k
                          << ", p.x, " << A << ".y);";
                }
                o << " }\n";
            }
            // keep each group's coefficients and partner reads next to its FMAs
            o << "    }\n    __builtin_amdgcn_sched_barrier(0);\n";
        }
        for (int rr = 0; rr < RC; rr++) {
            const int r = ch * RC + rr;
            const LdsSplit sp = lds_split(NT, r);
            o << "    {\n        const double2 ow = up2(la[(st ^ " << sp.low << "u) + " << sp.high << "u]);\n"
              << "        e = fma(ow.x, acc[" << rr << "].x, fma(ow.y, acc[" << rr << "].y, e));\n";
            o << "        const uint64_t gix = tile_index(tc, fb, " << (uint32_t)NT * r << "u + (uint32_t)tid);\n"
              << "        const float2 v = make_float2((float)(gw * acc[" << rr << "].x), (float)(gw * acc[" << rr
              << "].y));\n";
            if (pi == 0)
                o << "        pf[gix] = v;\n";
            else
                o << "        const float2 q = pf[gix];\n        pf[gix] = make_float2(q.x + v.x, q.y + v.y);\n";
            o << "    }\n";
        }
        o << "    }\n";
    }
    o << "    __syncthreads();\n"
         "    }\n"
         "    { const double v = wave_sum(e); if (lane == 0) red[wave] = v; }\n"
         "    __syncthreads();\n"
         "    if (tid == 0) {\n"
         "        double v = red[0];\n";
    for (int wv = 1; wv < NW; wv++) o << "        v += red[" << wv << "];\n";
    o << "        a.partial[(int64_t)(row * a.npass + " << pi << ") * a.wg_per_row + w] = v;\n"
         "    }\n"
         "}\n";
}

} // namespace

namespace {

// Terms per block of the expectation passes: one running sum (two VGPRs) per
// term of the block.
constexpr int kExpBlock = 16;
// observables of a generated expectation pass that keep register accumulators
constexpr int kSpecRegObs = 16;

// <psi|P|psi> of the pass's terms, for up to 16 observables: per thread 16
// amplitudes (the top four bits of the tile index).  The terms, grouped by
// their X mask on the tile, are taken in blocks; a block sweeps the 16
// registers with one running sum per term (s += Re or Im of
// conj(psi_l) psi_{l^x}, one partner read per group, the sign of the
// register bits of the term's Z mask written in) and then folds each sum into
// its observable's accumulator with the term's coefficient signed by the
// thread and tile bits of its Z mask.  A term whose X mask has a register bit
// visits each pair {l, l^x} once, with twice the coefficient.
// K: the set's observables.  Up to kSpecRegObs of them each keep an fp64
// accumulator in registers over the tile loop.  Larger sets run one tile per
// workgroup (the host launches one workgroup per tile) and keep per-wave
// sums in LDS: each block stores, per observable it touches, the wavefront
// sum of its terms' contributions in the wave's slot (lane 0; an observable
// met again in a later block of the pass is added to its slot).
void pauli_exp_pass(std::ostream &o, const PauliPass &pp, int pi, int K)
{
    const TileGeom &gm = pp.geom;
    const int t = gm.t, P = 16, tb = t - 4, NT = 1 << tb, NW = NT / 64;
    const bool lds_acc = K > kSpecRegObs;
    // observables of the pass, and the register accumulator of each
    std::vector<int> ks;
    for (const SpecTerm &tm : pp.terms)
        if (std::find(ks.begin(), ks.end(), tm.k) == ks.end()) ks.push_back(tm.k);
    std::sort(ks.begin(), ks.end());
    auto slot = [&](int k) { return (int)(std::find(ks.begin(), ks.end(), k) - ks.begin()); };
    const int NK = (int)ks.size();
    struct TT {
        uint32_t zlo, zhi;
        uint64_t zt;  // Z bits among the fixed bits, as tile-number bits
        double C;
        bool im;
        int kk;
    };
    std::map<uint32_t, std::vector<TT>> groups;
    for (const SpecTerm &tm : pp.terms) {
        const uint32_t xT = local_mask(gm, tm.x), zT = local_mask(gm, tm.z);
        const int ny = tm.ny & 3;
        const double chi = (__builtin_popcountll(tm.x & tm.z) & 1) ? -1.0 : 1.0;
        // <P> = Re(c' sum_l chi_z(l) conj(psi_l) psi_{l^x}), c' = coeff i^ny chi_z(x):
        // ny even: c' real, Re part; ny odd: c' = i b, -b times the Im part
        double C = (ny & 1) ? -(tm.coeff * (ny == 1 ? 1.0 : -1.0) * chi) : tm.coeff * (ny == 2 ? -1.0 : 1.0) * chi;
        // pairs {l, l^x} summed once when x has a register bit: twice the half
        if (xT >> tb) C *= 2.0;
        uint64_t zt = 0;
        for (int bb = 0, k = 0; bb < gm.n; bb++)
            if ((gm.fixed_mask >> bb) & 1) zt |= ((tm.z >> bb) & 1ull) << k++;
        groups[xT].push_back(TT{zT & (uint32_t)(NT - 1), zT >> tb, zt, C, (ny & 1) != 0, slot(tm.k)});
    }
    // blocks of at most kExpBlock terms; a group larger than what is left of
    // a block continues in the next one (its partner read again)
    struct Slice {
        uint32_t xT;
        std::vector<const TT *> tts;
        int first;  // running-sum index of its first term in the block
    };
    std::vector<std::vector<Slice>> blocks;
    {
        std::vector<Slice> cur;
        int cnt = 0;
        for (auto &g : groups)
            for (size_t i = 0; i < g.second.size();) {
                if (cnt == kExpBlock) {
                    blocks.push_back(std::move(cur));
                    cur.clear();
                    cnt = 0;
                }
                const size_t take = std::min(g.second.size() - i, (size_t)(kExpBlock - cnt));
                Slice sl{g.first, {}, cnt};
                for (size_t j = 0; j < take; j++) sl.tts.push_back(&g.second[i + j]);
                cur.push_back(std::move(sl));
                cnt += (int)take;
                i += take;
            }
        if (!cur.empty()) blocks.push_back(std::move(cur));
    }
    o << "extern \"C\" __global__ __launch_bounds__(" << NT << ", 4) void tq_pauli_" << pi
      << "(PauliSpecArgs a)\n{\n"
         "    extern __shared__ __align__(16) unsigned char smem[];\n"
         "    float2 *la = reinterpret_cast<float2 *>(smem);\n"
         "    uint64_t *hi_off = reinterpret_cast<uint64_t *>(la + "
      << (1 << t)
      << ");\n"
         "    double *red = reinterpret_cast<double *>(hi_off + "
      << (1 << gm.h)
      << ");\n"
         "    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;\n"
         "    const int row = blockIdx.x / a.wg_per_row, w = blockIdx.x % a.wg_per_row;\n"
         "    float2 *ps = const_cast<float2 *>(a.psi) + (int64_t)cget(a.rows, row) * a.row_stride;\n"
         "    build_hi_off(a.g, hi_off);\n"
         "    __syncthreads();  // hi_off complete before the first tile load\n"
         "    const TileCtx tc{hi_off, "
      << ((1u << gm.c) - 1) << "u, " << gm.c
      << "};\n"
         "    uint32_t tz = (uint32_t)tid;\n";
    if (lds_acc) {
        o << "    for (int i_ = tid; i_ < " << NW * K << "; i_ += " << NT << ") red[i_] = 0.0;\n"
             "    __syncthreads();\n";
    } else {
        for (int j = 0; j < NK; j++) o << "    double e" << j << " = 0.0;\n";
    }
    o << "    for (int64_t tile = w; tile < " << (1ll << (gm.n - t)) << "ll; tile += a.wg_per_row) {\n"
      << "    const uint64_t fb = pdep64((uint64_t)tile, " << gm.fixed_mask << "ull);\n"
      << "    tile_copy<true>(tc, la, ps, fb, " << (1 << t) << ");\n"
      << "    __syncthreads();\n";
    std::set<int> seen_k;  // LDS sums: observables already stored in this pass
    auto skipped = [&](uint32_t xT, int r) {
        const uint32_t xhi = xT >> tb;
        const int pivot = xhi ? 31 - __builtin_clz(xhi) : -1;
        return pivot >= 0 && ((r >> pivot) & 1);
    };
    for (const std::vector<Slice> &blk : blocks) {
        // the thread index and a zero made opaque anew per block: addresses
        // and signed coefficients are formed next to their use
        o << "    {\n    asm volatile(\"\" : \"+v\"(tz));\n"
          << "    uint32_t zc = 0u;\n    asm volatile(\"\" : \"+v\"(zc));\n"
          << "    const uint32_t vz = tz | ((uint32_t)tile << " << tb << ");\n"
          << "    const uint32_t st = sw(tz);\n";
        int nb = 0;
        for (const Slice &sl : blk) nb += (int)sl.tts.size();
        for (int j = 0; j < nb; j++) o << "    double s" << j << " = 0.0;\n";
        // rows by the low part of their swizzled offset: within a phase every
        // read of a slice goes through one base pointer, st ^ sw(x_lo) ^ low
        // (sw is linear over xor), with the rest of the offset immediate
        std::map<uint32_t, std::vector<int>> phases;
        for (int r = 0; r < P; r++) phases[lds_split(NT, r).low].push_back(r);
        for (auto &ph : phases) {
            const uint32_t lowr = ph.first;
            o << "    {\n    const float2 *lo = la + (st ^ " << lowr << "u);\n";
            for (size_t si = 0; si < blk.size(); si++) {
                const uint32_t xT = blk[si].xT, xhi = xT >> tb;
                if (!xT) continue;
                bool used = false;
                for (int r : ph.second) used |= !skipped(xT, r);
                if (!used) continue;
                const uint32_t c = host_sw(xT & (uint32_t)(NT - 1)) ^ lowr ^ lds_split(NT, xhi).low;
                o << "    const float2 *lp" << si << " = la + (st ^ " << c << "u);\n";
            }
            for (int r : ph.second) {
                o << "    {\n        const double2 o = up2(lo[" << lds_split(NT, r).high << "]);\n";
                for (size_t si = 0; si < blk.size(); si++) {
                    const Slice &sl = blk[si];
                    if (skipped(sl.xT, r)) continue;
                    bool any_re = false, any_im = false;
                    for (const TT *tt : sl.tts) (tt->im ? any_im : any_re) = true;
                    o << "        {\n";
                    if (sl.xT) {
                        o << "        const double2 p = up2(lp" << si << "[" << lds_split(NT, r ^ (sl.xT >> tb)).high
                          << "]);\n";
                        if (any_re) o << "        const double re = fma(o.x, p.x, o.y * p.y);\n";
                        if (any_im) o << "        const double im = fma(o.x, p.y, -o.y * p.x);\n";
                    } else {
                        o << "        const double re = fma(o.x, o.x, o.y * o.y);\n";
                    }
                    for (size_t j = 0; j < sl.tts.size(); j++) {
                        const TT &tt = *sl.tts[j];
                        const bool neg = __builtin_popcount(tt.zhi & (uint32_t)r) & 1;
                        o << "        s" << sl.first + (int)j << (neg ? " -= " : " += ") << (tt.im ? "im" : "re")
                          << ";\n";
                    }
                    o << "        }\n";
                }
                o << "    }\n";
            }
            o << "    }\n";
        }
        // fold: the coefficient's sign bit flipped by the parity of the
        // thread and tile bits of the term's Z mask
        auto coef = [&](const TT &tt) {
            const uint64_t m = (uint64_t)tt.zlo | (tt.zt << tb);
            uint64_t cb;
            std::memcpy(&cb, &tt.C, sizeof cb);
            std::string c = "__hiloint2double((int)(" + std::to_string((uint32_t)(cb >> 32)) + "u ^ ";
            if (!m) c += "zc";
            else c += "((uint32_t)(__popc(vz & " + std::to_string(m) + "u) & 1) << 31)";
            return c + "), (int)(" + std::to_string((uint32_t)cb) + "u ^ zc))";
        };
        if (!lds_acc) {
            for (const Slice &sl : blk)
                for (size_t j = 0; j < sl.tts.size(); j++) {
                    const TT &tt = *sl.tts[j];
                    o << "    e" << tt.kk << " = fma(" << coef(tt) << ", s" << sl.first + (int)j << ", e" << tt.kk
                      << ");\n";
                }
        } else {
            // per observable of the block (at most 16): its terms'
            // contributions summed into u_m; then a reduce-scatter over the
            // lane bits 0..3 (lane l keeps u_{T(l)}, T(l) = 8 l0 + 4 l1 +
            // 2 l2 + l3, the sum over its 16 lanes) and the two row
            // exchanges leave the wavefront sum of u_m in lanes l < 16 with
            // T(l) = m, which store it in (or, met before, add it to) the
            // wave's slot of that observable
            std::map<int, std::vector<std::pair<const TT *, int>>> by_k;
            for (const Slice &sl : blk)
                for (size_t j = 0; j < sl.tts.size(); j++) by_k[ks[sl.tts[j]->kk]].push_back({sl.tts[j], sl.first + (int)j});
            std::vector<int> kms;
            o << "    {\n";
            for (auto &kv : by_k) {
                const int m = (int)kms.size();
                kms.push_back(kv.first);
                o << "      double u" << m << " = 0.0;\n";
                for (auto &tj : kv.second) o << "      u" << m << " = fma(" << coef(*tj.first) << ", s" << tj.second << ", u" << m << ");\n";
            }
            int M = (int)kms.size();  // entries u_0 .. u_{M-1} not known to be zero
            for (int step = 0, half = 8; step < 4; step++, half /= 2) {
                const int bitv = 1 << step;
                auto u = [&](int q) { return q < M ? "u" + std::to_string(q) : std::string("0.0"); };
                for (int i = 0; i < std::min(M, half); i++)
                    o << "      { const bool h_ = (lane & " << bitv << ") != 0; const double k_ = h_ ? " << u(i + half)
                      << " : " << u(i) << ", x_ = h_ ? " << u(i) << " : " << u(i + half) << "; u" << i
                      << " = k_ + __shfl_xor(x_, " << bitv << ", 64); }\n";
                M = std::min(M, half);
            }
            o << "      u0 += __shfl_xor(u0, 16, 64);\n"
                 "      u0 += __shfl_xor(u0, 32, 64);\n"
                 "      const int t_ = ((lane & 1) << 3) | ((lane & 2) << 1) | ((lane >> 1) & 2) | ((lane >> 3) & 1);\n"
                 "      if (lane < 16) {\n"
                 "        switch (t_) {\n";
            for (int m = 0; m < (int)kms.size(); m++) {
                o << "        case " << m << ": red[wave * " << K << " + " << kms[m] << "] "
                  << (seen_k.count(kms[m]) ? "+=" : "=") << " u0; break;\n";
                seen_k.insert(kms[m]);
            }
            o << "        default: break;\n        }\n      }\n    }\n";
        }
        o << "    }\n    __builtin_amdgcn_sched_barrier(0);\n";
    }
    o << "    __syncthreads();\n"
         "    }\n";
    if (lds_acc) {
        // the per-wave sums, in wave order
        o << "    double *out = a.partial + ((int64_t)(row * a.npass + " << pi
          << ") * a.wg_per_row + w) * a.k_count;\n"
             "    for (int k = tid; k < a.k_count; k += "
          << NT << ") {\n        double v = red[k];\n";
        for (int wv = 1; wv < NW; wv++) o << "        v += red[" << wv * K << " + k];\n";
        o << "        out[k] = v;\n    }\n}\n";
        return;
    }
    // fixed-order reduction: waves, then the wave sums
    for (int j = 0; j < NK; j++)
        o << "    { const double v = wave_sum(e" << j << "); if (lane == 0) red[wave * " << NK << " + " << j << "] = v; }\n";
    o << "    __syncthreads();\n"
         "    double *out = a.partial + ((int64_t)(row * a.npass + "
      << pi
      << ") * a.wg_per_row + w) * a.k_count;\n"
         "    for (int k = tid; k < a.k_count; k += "
      << NT
      << ") {\n"
         "        double v = 0.0;\n"
         "        switch (k) {\n";
    for (int j = 0; j < NK; j++) {
        o << "        case " << ks[j] << ": v = red[" << j << "]";
        for (int wv = 1; wv < NW; wv++) o << "; v += red[" << wv * NK + j << "]";
        o << "; break;\n";
    }
    o << "        default: break;\n"
         "        }\n"
         "        out[k] = v;\n"
         "    }\n"
         "}\n";
}

} // namespace

std::string pauli_spec_source(const std::vector<PauliPass> &passes, int K)
{
    std::ostringstream o;
    o << kHead;
    for (size_t pi = 0; pi < passes.size(); pi++) pauli_exp_pass(o, passes[pi], (int)pi, K);
    o << "} // namespace tq\n";
    return o.str();
}

namespace {

struct Module {
    hipModule_t mod = nullptr;
    std::map<std::string, hipFunction_t> fn;
};

std::mutex g_mu;
// (device, kernel source) -> loaded module; kept until the process ends
std::map<std::pair<int, std::string>, Module> g_cache;
int g_compiled = 0;

// ---------------------------------------------------------- code cache
// Compiled code objects are kept on disk, keyed by a 128-bit hash of
// everything that determines them (the shared device code, the kernel
// source, the offload target and the compiler options), so that a circuit
// structure compiles once per machine.  Directory: $TQ_CACHE_DIR, else
// $XDG_CACHE_HOME/tq-kernels, else $HOME/.cache/tq-kernels; TQ_CACHE_DIR=""
// (empty) turns the cache off.  Files are written under a temporary name
// and renamed, so that concurrent processes never read a partial file.
constexpr int kCompileOpts = 7;
const char *const kOptsTail[] = {"-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"};

std::string cache_dir()
{
    const char *d = std::getenv("TQ_CACHE_DIR");
    if (d) return d;
    if ((d = std::getenv("XDG_CACHE_HOME")) && *d) return std::string(d) + "/tq-kernels";
    if ((d = std::getenv("HOME")) && *d) return std::string(d) + "/.cache/tq-kernels";
    return "";
}

// FNV-1a over the bytes, in two independent 64-bit lanes
std::string hash128(const std::string &text)
{
    uint64_t a = 1469598103934665603ull, b = 0x9e3779b97f4a7c15ull;
    for (unsigned char ch : text) {
        a = (a ^ ch) * 1099511628211ull;
        b = (b ^ ch) * 0x100000001b3ull ^ (b >> 29);
    }
    char buf[40];
    snprintf(buf, sizeof buf, "%016llx%016llx", (unsigned long long)a, (unsigned long long)b);
    return buf;
}

bool cache_read(const std::string &path, std::vector<char> *code)
{
    std::ifstream f(path, std::ios::binary);
    if (!f) return false;
    std::vector<char> v((std::istreambuf_iterator<char>(f)), std::istreambuf_iterator<char>());
    if (v.empty()) return false;
    code->swap(v);
    return true;
}

void cache_write(const std::string &dir, const std::string &path, const std::vector<char> &code)
{
    // mkdir -p
    for (size_t i = 1; i <= dir.size(); i++)
        if (i == dir.size() || dir[i] == '/') mkdir(dir.substr(0, i).c_str(), 0755);
    const std::string tmp = path + ".tmp" + std::to_string((long)getpid()) + "_" +
                            std::to_string((unsigned long long)std::hash<std::thread::id>()(std::this_thread::get_id()));
    {
        std::ofstream f(tmp, std::ios::binary);
        if (!f) return;
        f.write(code.data(), (std::streamsize)code.size());
        if (!f) {
            std::remove(tmp.c_str());
            return;
        }
    }
    if (std::rename(tmp.c_str(), path.c_str()) != 0) std::remove(tmp.c_str());
}

std::atomic<int> g_disk_hits{0};

// Compile the kernel source `body` for offload target `target` into a code
// object (or read it from the code cache).
hipError_t compile_code(const std::string &body, const std::string &target, std::vector<char> *code,
                        std::string *log)
{
    const std::string src = std::string(kPrelude) + "\n" + body;
    const std::string arch = "--offload-arch=" + target;
    std::string key = src + "\n//" + arch;
    for (const char *o : kOptsTail) key += std::string(" ") + o;
    const std::string dir = cache_dir();
    const std::string path = dir.empty() ? "" : dir + "/" + hash128(key) + "_" + target + ".co";
    if (!path.empty() && cache_read(path, code)) {
        g_disk_hits++;
        return hipSuccess;
    }
    hiprtcProgram prog;
    if (hiprtcCreateProgram(&prog, src.c_str(), "tq_spec.hip", 0, nullptr, nullptr) != HIPRTC_SUCCESS) {
        *log = "hiprtcCreateProgram failed";
        return hipErrorInvalidSource;
    }
    // the same code generation flags as the precompiled kernels
    const char *opts[kCompileOpts] = {arch.c_str()};
    for (int i = 1; i < kCompileOpts; i++) opts[i] = kOptsTail[i - 1];
    const hiprtcResult r = hiprtcCompileProgram(prog, kCompileOpts, opts);
    if (r != HIPRTC_SUCCESS) {
        size_t n = 0;
        hiprtcGetProgramLogSize(prog, &n);
        std::string text(n, '\0');
        if (n) hiprtcGetProgramLog(prog, &text[0]);
        *log = "specialised kernel: " + std::string(hiprtcGetErrorString(r)) + "\n" + text;
        hiprtcDestroyProgram(&prog);
        return hipErrorInvalidSource;
    }
    size_t size = 0;
    hiprtcGetCodeSize(prog, &size);
    code->resize(size);
    hiprtcGetCode(prog, code->data());
    hiprtcDestroyProgram(&prog);
    if (!path.empty()) cache_write(dir, path, *code);
    return hipSuccess;
}

// Compile several sources for one target at once, one thread each (at most
// the host's hardware threads, up to 16, at a time).
hipError_t compile_many(const std::vector<const std::string *> &bodies, const std::string &target,
                        std::vector<std::vector<char>> *codes, std::string *log)
{
    codes->assign(bodies.size(), {});
    std::vector<hipError_t> err(bodies.size(), hipSuccess);
    std::vector<std::string> logs(bodies.size());
    const size_t width = std::max<size_t>(1, std::min<size_t>(16, std::thread::hardware_concurrency()));
    for (size_t b0 = 0; b0 < bodies.size(); b0 += width) {
        std::vector<std::thread> th;
        for (size_t i = b0; i < std::min(bodies.size(), b0 + width); i++)
            th.emplace_back([&, i] { err[i] = compile_code(*bodies[i], target, &(*codes)[i], &logs[i]); });
        for (auto &t : th) t.join();
    }
    for (size_t i = 0; i < bodies.size(); i++)
        if (err[i] != hipSuccess) {
            *log = logs[i];
            return err[i];
        }
    return hipSuccess;
}

// The kernels `names` of source `body` on the current device: compiled and
// loaded on first use.
hipError_t get_kernels(const std::string &body, const std::vector<std::string> &names,
                       std::vector<hipFunction_t> *fns, std::string *log)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> l(g_mu);
    auto key = std::make_pair(dev, body);
    auto it = g_cache.find(key);
    if (it == g_cache.end()) {
        hipDeviceProp_t prop;
        e = hipGetDeviceProperties(&prop, dev);
        if (e != hipSuccess) return e;
        std::vector<char> code;
        e = compile_code(body, prop.gcnArchName, &code, log);
        if (e != hipSuccess) return e;
        Module m;
        e = hipModuleLoadData(&m.mod, code.data());
        if (e != hipSuccess) return e;
        it = g_cache.emplace(std::move(key), std::move(m)).first;
        g_compiled++;
    }
    fns->clear();
    for (const std::string &n : names) {
        auto f = it->second.fn.find(n);
        if (f == it->second.fn.end()) {
            hipFunction_t fn;
            e = hipModuleGetFunction(&fn, it->second.mod, n.c_str());
            if (e != hipSuccess) return e;
            f = it->second.fn.emplace(n, fn).first;
        }
        fns->push_back(f->second);
    }
    return hipSuccess;
}

// Load the sources `bodies` on the current device, compiling (in parallel)
// those not loaded yet.
hipError_t load_all(const std::vector<std::string> &bodies, std::string *log)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::vector<const std::string *> missing;
    {
        std::lock_guard<std::mutex> l(g_mu);
        for (const std::string &b : bodies)
            if (!g_cache.count(std::make_pair(dev, b))) missing.push_back(&b);
    }
    if (missing.empty()) return hipSuccess;
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) return e;
    std::vector<std::vector<char>> codes;
    e = compile_many(missing, prop.gcnArchName, &codes, log);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> l(g_mu);
    for (size_t i = 0; i < missing.size(); i++) {
        auto key = std::make_pair(dev, *missing[i]);
        if (g_cache.count(key)) continue;
        Module m;
        e = hipModuleLoadData(&m.mod, codes[i].data());
        if (e != hipSuccess) return e;
        g_cache.emplace(std::move(key), std::move(m));
        g_compiled++;
    }
    return hipSuccess;
}

// The pass kernels of group g are compiled as programs of up to
// kChunkPasses passes each (forward and reverse separately).  The run-time
// compiler serialises compilations within a process (measured: 16 threads
// take as long as one), so a structure's passes form one program each way,
// which parses the shared device code once.  Reverse passes only run for
// gradients: a structure without symbolic parameters never launches them,
// and gets none.
constexpr int kChunkPasses = 256;
int fwd_chunks(const Group &g) { return ((int)g.fwd.size() + kChunkPasses - 1) / kChunkPasses; }
int rev_chunks(const Group &g) { return g.n_gslots > 0 ? ((int)g.rev.size() + kChunkPasses - 1) / kChunkPasses : 0; }

std::string pass_chunk(const Group &g, int chunk)
{
    std::string body = kHead;
    const int nf = fwd_chunks(g);
    const bool rev = chunk >= nf;
    const int c = rev ? chunk - nf : chunk;
    const int np = rev ? (int)g.rev.size() : (int)g.fwd.size();
    for (int pi = c * kChunkPasses; pi < std::min(np, (c + 1) * kChunkPasses); pi++)
        body += rev ? rev_pass_kernel_source(g, pi) : pass_kernel_source(g, pi);
    return body + "} // namespace tq\n";
}

std::vector<std::string> pass_chunks(const Group &g)
{
    std::vector<std::string> v;
    for (int c = 0; c < fwd_chunks(g) + rev_chunks(g); c++) v.push_back(pass_chunk(g, c));
    return v;
}

template <class Args>
hipError_t launch(hipFunction_t fn, const Args &a, unsigned grid, size_t lds, hipStream_t s, const char *prof_name,
                  unsigned threads = kThreads)
{
    if (lds > 65536) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(fn),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    Args args = a;
    void *params[] = {&args};
    ProfScope ps(prof_name, s);
    return hipModuleLaunchKernel(fn, grid, 1, 1, threads, 1, 1, (unsigned)lds, s, params, nullptr);
}

// Kernel `name` of the program whose source `src()` generates, through the
// caller's memo (slot `slot` of `nslots`) when it has one: the source is
// generated and looked up only the first time on a device.
template <class Src>
hipError_t memo_kernel(SpecMemo *memo, size_t slot, size_t nslots, Src &&src, const std::string &name,
                       hipFunction_t *fn, std::string *log)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (memo && memo->dev == dev && slot < memo->fn.size() && memo->fn[slot]) {
        *fn = memo->fn[slot];
        return hipSuccess;
    }
    std::vector<hipFunction_t> fns;
    e = get_kernels(src(), {name}, &fns, log);
    if (e != hipSuccess) return e;
    *fn = fns[0];
    if (memo) {
        if (memo->dev != dev || memo->fn.size() != nslots) {
            memo->dev = dev;
            memo->fn.assign(nslots, nullptr);
            memo->slots = -1;
        }
        if (slot < nslots) memo->fn[slot] = fns[0];
    }
    return hipSuccess;
}

// Forward or reverse pass kernel `pass` of group g: on the first request on
// a device every chunk of the group is compiled (in parallel) and loaded.
hipError_t pass_kernel(const Group &g, bool rev, int pass, hipFunction_t *fn, std::string *log, SpecMemo *memo)
{
    const size_t slot = (rev ? g.fwd.size() : 0) + (size_t)pass, nslots = g.fwd.size() + g.rev.size();
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (!(memo && memo->dev == dev && slot < memo->fn.size() && memo->fn[slot])) {
        e = load_all(pass_chunks(g), log);
        if (e != hipSuccess) return e;
    }
    const int chunk = rev ? fwd_chunks(g) + pass / kChunkPasses : pass / kChunkPasses;
    return memo_kernel(memo, slot, nslots, [&] { return pass_chunk(g, chunk); },
                       (rev ? "tq_rev_" : "tq_fwd_") + N(pass), fn, log);
}

} // namespace

hipError_t launch_resident_spec(const Group &g, const ResArgs &a, int nrows, size_t lds, hipStream_t s,
                                std::string *log, SpecMemo *memo)
{
    if (nrows <= 0) return hipSuccess;
    hipFunction_t fn;
    hipError_t e = memo_kernel(memo, 0, 1, [&] { return resident_source(g); }, "tq_resident_spec", &fn, log);
    if (e != hipSuccess) return e;
    return launch(fn, a, nrows, lds, s, "resident", resident_threads(g));
}

hipError_t launch_pass_spec(const Group &g, int pass, const PassArgs &a, int nrows, hipStream_t s,
                            std::string *log, SpecMemo *memo)
{
    if (nrows <= 0) return hipSuccess;
    hipFunction_t fn;
    hipError_t e = pass_kernel(g, false, pass, &fn, log, memo);
    if (e != hipSuccess) return e;
    const size_t lds = pass_lds_bytes(a.g, a.product_init != 0, a.mat_end - a.mat_begin);
    return launch(fn, a, nrows * a.wg_per_row, lds, s, "pass");
}

std::string hphi_spec_source(const std::vector<PauliPass> &passes)
{
    std::ostringstream o;
    o << kHead;
    for (size_t pi = 0; pi < passes.size(); pi++) hphi_pass(o, passes[pi], (int)pi);
    o << "} // namespace tq\n";
    return o.str();
}

hipError_t launch_hphi_spec(const std::string &src, int pass, const HPhiArgs &a, int nrows, hipStream_t s,
                            std::string *log, SpecMemo *memo)
{
    if (nrows <= 0) return hipSuccess;
    hipFunction_t fn;
    hipError_t e = memo_kernel(memo, (size_t)pass, (size_t)a.npass, [&] { return src; }, "tq_hphi_" + N(pass), &fn, log);
    if (e != hipSuccess) return e;
    return launch(fn, a, nrows * a.wg_per_row, pauli_spec_lds_bytes(a.g, 16), s, "pauli", pauli_spec_threads(a.g));
}

hipError_t launch_pauli_spec(const std::string &src, int pass, const PauliSpecArgs &a, int nrows, hipStream_t s,
                             std::string *log, SpecMemo *memo)
{
    if (nrows <= 0) return hipSuccess;
    hipFunction_t fn;
    hipError_t e = memo_kernel(memo, (size_t)pass, (size_t)a.npass, [&] { return src; }, "tq_pauli_" + N(pass), &fn,
                               log);
    if (e != hipSuccess) return e;
    return launch(fn, a, nrows * a.wg_per_row, pauli_spec_lds_bytes(a.g, a.k_count), s, "pauli",
                  pauli_spec_threads(a.g));
}

int pauli_spec_slots(const std::string &src, const TileGeom &g, int K, std::string *log, SpecMemo *memo)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (memo && memo->dev == dev && memo->slots >= 0) return memo->slots;
    std::vector<hipFunction_t> fn;
    if (get_kernels(src, {"tq_pauli_0"}, &fn, log) != hipSuccess) return 0;
    int per_cu = 0, cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    if (pauli_spec_lds_bytes(g, K) > 65536 &&
        hipFuncSetAttribute(reinterpret_cast<const void *>(fn[0]), hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)pauli_spec_lds_bytes(g, K)) != hipSuccess)
        return 0;
    if (hipModuleOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn[0], pauli_spec_threads(g),
                                                           pauli_spec_lds_bytes(g, K)) != hipSuccess)
        return 0;
    if (memo && memo->dev == dev) memo->slots = per_cu * cus;
    return per_cu * cus;
}

hipError_t launch_rev_pass_spec(const Group &g, int pass, const RevArgs &a, int nrows, hipStream_t s,
                                std::string *log, SpecMemo *memo)
{
    if (nrows <= 0) return hipSuccess;
    hipFunction_t fn;
    hipError_t e = pass_kernel(g, true, pass, &fn, log, memo);
    if (e != hipSuccess) return e;
    return launch(fn, a, nrows * a.wg_per_row, rev_pass_lds_bytes(a), s, "rev_pass");
}

hipError_t prepare_spec(const Group &g, bool resident, const char *target, std::string *log)
{
    const std::vector<std::string> bodies = resident ? std::vector<std::string>{resident_source(g)} : pass_chunks(g);
    if (target) {
        std::vector<const std::string *> ptrs;
        for (const std::string &b : bodies) ptrs.push_back(&b);
        std::vector<std::vector<char>> codes;
        return compile_many(ptrs, target, &codes, log);
    }
    return load_all(bodies, log);
}

int spec_disk_cache_hits() { return g_disk_hits.load(); }

int spec_kernels_compiled()
{
    std::lock_guard<std::mutex> l(g_mu);
    return g_compiled;
}

} // namespace tq
