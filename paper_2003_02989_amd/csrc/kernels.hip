// kernels.hip -- HIP kernels of libtq for CDNA4 (gfx950), wave64.
//
// State vectors are complex64 (float2) rows of 2^n amplitudes in HBM.  Every
// sweep over a state is a tile kernel: a 256-thread workgroup stages tiles of
// 2^t amplitudes in LDS (t index bits = the `c` lowest bits, so that each
// wavefront reads contiguous runs, plus `h` high bits), works on them and
// writes them back.  Gate matrices are resolved from the symbol values and
// pre-multiplied (fused) in float64 by a separate builder kernel and rounded
// once to complex64.  All reductions are two-stage and fixed-order (no
// floating-point atomics), so every output is bitwise reproducible.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"

namespace tq {

// ------------------------------------------------------------ small helpers
// fp64 arithmetic on complex64 amplitudes: gate matrices stay in float64 and
// every product is formed in float64; only the stored amplitude is rounded
// Read-only tables (ops, stages, term lists) are read through the constant
// address space: with a uniform index the load becomes a scalar-cache load
// instead of a vector memory load that the wave has to wait for.
template <class T> __device__ __forceinline__ T cget(const T *p, int64_t i)
{
    static_assert(sizeof(T) % 4 == 0, "tables are read in 32-bit words");
    typedef const __attribute__((address_space(4))) uint32_t cword;
    cword *q = (cword *)(p + i);
    T v;
    uint32_t *d = reinterpret_cast<uint32_t *>(&v);
#pragma unroll
    for (int k = 0; k < (int)(sizeof(T) / 4); k++) d[k] = q[k];
    return v;
}

__device__ __forceinline__ double2 up2(float2 a) { return make_double2((double)a.x, (double)a.y); }
__device__ __forceinline__ float2 down2(double2 a) { return make_float2((float)a.x, (float)a.y); }
__device__ __forceinline__ double2 zmul(double2 a, double2 b)
{
    return make_double2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
__device__ __forceinline__ double2 zmul2(double2 m0, double2 a0, double2 m1, double2 a1)
{
    return make_double2(m0.x * a0.x - m0.y * a0.y + m1.x * a1.x - m1.y * a1.y,
                        m0.x * a0.y + m0.y * a0.x + m1.x * a1.y + m1.y * a1.x);
}
__device__ __forceinline__ double2 zadd(double2 a, double2 b) { return make_double2(a.x + b.x, a.y + b.y); }
// Re(conj(a) b)
__device__ __forceinline__ double zdotr(double2 a, double2 b) { return a.x * b.x + a.y * b.y; }

// LDS position of tile element i: an XOR swizzle that keeps runs of 32
// consecutive elements on distinct bank pairs and spreads strided stage
// gathers (lanes 2^r elements apart) over the banks as well
__device__ __forceinline__ uint32_t sw(uint32_t i) { return i ^ ((i >> 5) & 31u); }

// insert a zero bit at position k of p
__device__ __forceinline__ uint32_t ins0(uint32_t p, int k) { return ((p >> k) << (k + 1)) | (p & ((1u << k) - 1)); }

// deposit the low bits of v at the set bits of mask
__device__ uint64_t pdep64(uint64_t v, uint64_t mask)
{
    uint64_t r = 0;
    for (int k = 0; mask; k++) {
        uint64_t low = mask & (~mask + 1);
        if ((v >> k) & 1) r |= low;
        mask ^= low;
    }
    return r;
}

// Wavefront sum of a double, in the VALU: DPP quad swaps and row mirrors
// sum each row of 16 lanes, then the four row sums are read out and added
// (in the same order in every lane, so every lane returns the same value).
template <int kCtrl> __device__ __forceinline__ double dpp_mov(double v)
{
    const long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_mov_dpp((int)b, kCtrl, 0xf, 0xf, false);
    const int hi = __builtin_amdgcn_mov_dpp((int)(b >> 32), kCtrl, 0xf, 0xf, false);
    return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}
__device__ __forceinline__ double read_lane(double v, int lane)
{
    const long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_readlane((int)b, lane), hi = __builtin_amdgcn_readlane((int)(b >> 32), lane);
    return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}
__device__ __forceinline__ double wave_sum(double v)
{
    v += dpp_mov<0xb1>(v);   // quad_perm [1,0,3,2]: lane ^ 1
    v += dpp_mov<0x4e>(v);   // quad_perm [2,3,0,1]: lane ^ 2
    v += dpp_mov<0x141>(v);  // row_half_mirror: the other quad of the half row
    v += dpp_mov<0x140>(v);  // row_mirror: the other half of the row
    return (read_lane(v, 0) + read_lane(v, 16)) + (read_lane(v, 32) + read_lane(v, 48));
}

// parity of popcount
__device__ __forceinline__ int par64(uint64_t v) { return __popcll(v) & 1; }
__device__ __forceinline__ int par32(uint32_t v) { return __popc(v) & 1; }

// ---------------------------------------------------- gate matrices (fp64)
// Closed forms of the opcode set, written from the gate definitions: for an
// involutory generator G, G^t = (1+w)/2 I + (1-w)/2 G with w = e^{i pi t}
// (the phase convention e^{i pi t/2}(cos(pi t/2) I - i sin(pi t/2) G)), and a
// rotation exp(-i theta G / 2) = cos(theta/2) I - i sin(theta/2) G.
struct cd {
    double x, y;
};
__device__ __forceinline__ cd C(double x, double y) { return cd{x, y}; }
__device__ __forceinline__ cd cdmul(cd a, cd b) { return cd{a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x}; }
__device__ __forceinline__ cd cdadd(cd a, cd b) { return cd{a.x + b.x, a.y + b.y}; }
__device__ __forceinline__ cd cdscale(cd a, double s) { return cd{a.x * s, a.y * s}; }

// m: row-major d x d, zero-initialised by the caller
__device__ __forceinline__ int gate_matrix_dev(int op, const double *eta, const double *ex, int form, cd *m)
{
    const double r = 0.70710678118654752440;
    double c, s;
    switch (op) {
    case OP_H: m[0] = C(r, 0); m[1] = C(r, 0); m[2] = C(r, 0); m[3] = C(-r, 0); return 2;
    case OP_X: m[1] = C(1, 0); m[2] = C(1, 0); return 2;
    case OP_Y: m[1] = C(0, -1); m[2] = C(0, 1); return 2;
    case OP_Z: m[0] = C(1, 0); m[3] = C(-1, 0); return 2;
    case OP_RX:
        sincos(eta[0] * 0.5, &s, &c);
        m[0] = C(c, 0); m[1] = C(0, -s); m[2] = C(0, -s); m[3] = C(c, 0); return 2;
    case OP_RY:
        sincos(eta[0] * 0.5, &s, &c);
        m[0] = C(c, 0); m[1] = C(-s, 0); m[2] = C(s, 0); m[3] = C(c, 0); return 2;
    case OP_RZ:
        sincos(eta[0] * 0.5, &s, &c);
        m[0] = C(c, -s); m[3] = C(c, s); return 2;
    case OP_XPOW: case OP_YPOW: case OP_ZPOW: case OP_SQRTX: case OP_SQRTY: case OP_SQRTW: {
        double t = (op == OP_SQRTX || op == OP_SQRTY || op == OP_SQRTW) ? 0.5 : eta[0];
        sincospi(t, &s, &c);
        cd a = C(0.5 * (1 + c), 0.5 * s);   // (1 + w) / 2
        cd bq = C(0.5 * (1 - c), -0.5 * s); // (1 - w) / 2
        if (op == OP_ZPOW) { m[0] = C(1, 0); m[3] = C(c, s); return 2; }
        m[0] = a; m[3] = a;
        if (op == OP_XPOW || op == OP_SQRTX) { m[1] = bq; m[2] = bq; }
        else if (op == OP_YPOW || op == OP_SQRTY) { m[1] = cdmul(bq, C(0, -1)); m[2] = cdmul(bq, C(0, 1)); }
        else { m[1] = cdmul(bq, C(r, -r)); m[2] = cdmul(bq, C(r, r)); } // W = [[0, e^{-i pi/4}], [e^{i pi/4}, 0]]
        return 2;
    }
    case OP_CZ:
        m[0] = m[5] = m[10] = C(1, 0); m[15] = C(-1, 0); return 4;
    case OP_CZPOW:
        sincospi(eta[0], &s, &c);
        m[0] = m[5] = m[10] = C(1, 0); m[15] = C(c, s); return 4;
    case OP_CNOT:
        if (form == FORM_CBLOCK) { m[1] = m[2] = C(1, 0); return 2; }
        m[0] = m[5] = C(1, 0); m[11] = m[14] = C(1, 0); return 4;
    case OP_CNOTPOW: {
        sincospi(eta[0], &s, &c);
        cd a = C(0.5 * (1 + c), 0.5 * s), bq = C(0.5 * (1 - c), -0.5 * s);
        if (form == FORM_CBLOCK) { m[0] = m[3] = a; m[1] = m[2] = bq; return 2; }
        m[0] = m[5] = C(1, 0); m[10] = m[15] = a; m[11] = m[14] = bq; return 4;
    }
    case OP_XXPOW: case OP_YYPOW: {
        sincospi(eta[0], &s, &c);
        cd a = C(0.5 * (1 + c), 0.5 * s), bq = C(0.5 * (1 - c), -0.5 * s);
        m[0] = m[5] = m[10] = m[15] = a;
        if (op == OP_XXPOW) { m[3] = m[6] = m[9] = m[12] = bq; }
        else { m[3] = m[12] = cdscale(bq, -1); m[6] = m[9] = bq; } // YY: -|11><00| - |00><11| + |10><01| + |01><10|
        return 4;
    }
    case OP_ZZPOW:
        sincospi(eta[0], &s, &c);
        m[0] = m[15] = C(1, 0); m[5] = m[10] = C(c, s); return 4;
    case OP_RZZ:
        sincos(eta[0] * 0.5, &s, &c);
        m[0] = m[15] = C(c, -s); m[5] = m[10] = C(c, s); return 4;
    case OP_FSIM:
        sincos(eta[0], &s, &c);
        m[0] = C(1, 0); m[5] = m[10] = C(c, 0); m[6] = m[9] = C(0, -s);
        sincos(eta[1], &s, &c);
        m[15] = C(c, -s); return 4;
    case OP_SWAP:
        m[0] = m[6] = m[9] = m[15] = C(1, 0); return 4;
    case OP_MATRIX1:
        for (int i = 0; i < 4; i++) m[i] = C(ex[2 * i], ex[2 * i + 1]);
        return 2;
    case OP_MATRIX2:
        for (int i = 0; i < 16; i++) m[i] = C(ex[2 * i], ex[2 * i + 1]);
        return 4;
    }
    return 0;
}

// derivative with respect to parameter `which` (m zero-initialised)
__device__ __forceinline__ int gate_deriv_dev(int op, const double *eta, int which, int form, cd *m)
{
    double c, s;
    const double pi = 3.14159265358979323846;
    switch (op) {
    case OP_RX:
        sincos(eta[0] * 0.5, &s, &c);
        m[0] = C(-0.5 * s, 0); m[1] = C(0, -0.5 * c); m[2] = C(0, -0.5 * c); m[3] = C(-0.5 * s, 0); return 2;
    case OP_RY:
        sincos(eta[0] * 0.5, &s, &c);
        m[0] = C(-0.5 * s, 0); m[1] = C(-0.5 * c, 0); m[2] = C(0.5 * c, 0); m[3] = C(-0.5 * s, 0); return 2;
    case OP_RZ:
        sincos(eta[0] * 0.5, &s, &c);
        m[0] = C(-0.5 * s, -0.5 * c); m[3] = C(-0.5 * s, 0.5 * c); return 2;
    case OP_RZZ:
        sincos(eta[0] * 0.5, &s, &c);
        m[0] = m[15] = C(-0.5 * s, -0.5 * c); m[5] = m[10] = C(-0.5 * s, 0.5 * c); return 4;
    case OP_XPOW: case OP_YPOW: case OP_ZPOW: case OP_CZPOW: case OP_CNOTPOW:
    case OP_XXPOW: case OP_YYPOW: case OP_ZZPOW: {
        // d/dt G^t = (i pi w / 2)(I - G), w = e^{i pi t}
        sincospi(eta[0], &s, &c);
        cd k = C(-0.5 * pi * s, 0.5 * pi * c);  // i pi w / 2
        cd mk = cdscale(k, -1);
        switch (op) {
        case OP_XPOW: m[0] = m[3] = k; m[1] = m[2] = mk; return 2;
        case OP_YPOW: m[0] = m[3] = k; m[1] = cdmul(mk, C(0, -1)); m[2] = cdmul(mk, C(0, 1)); return 2;
        case OP_ZPOW: m[3] = cdscale(k, 2); return 2;
        case OP_CZPOW: m[15] = cdscale(k, 2); return 4;
        case OP_CNOTPOW:
            if (form == FORM_CBLOCK) { m[0] = m[3] = k; m[1] = m[2] = mk; return 2; }
            m[10] = m[15] = k; m[11] = m[14] = mk; return 4;
        case OP_XXPOW: m[0] = m[5] = m[10] = m[15] = k; m[3] = m[6] = m[9] = m[12] = mk; return 4;
        case OP_YYPOW: m[0] = m[5] = m[10] = m[15] = k; m[3] = m[12] = k; m[6] = m[9] = mk; return 4;
        case OP_ZZPOW: m[5] = m[10] = cdscale(k, 2); return 4;
        }
        return 0;
    }
    case OP_FSIM:
        if (which == 0) {
            sincos(eta[0], &s, &c);
            m[5] = m[10] = C(-s, 0); m[6] = m[9] = C(0, -c);
        } else {
            sincos(eta[1], &s, &c);
            m[15] = C(-s, -c);  // -i e^{-i phi}
        }
        return 4;
    }
    return 0;
}

// permutation of a 4x4 two-qubit matrix for reversed qubit order (|ab> -> |ba>)
__device__ __forceinline__ void swap_qubits4(cd *m)
{
    cd t[16];
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const int pi = (i == 1) ? 2 : (i == 2) ? 1 : i, pj = (j == 1) ? 2 : (j == 2) ? 1 : j;
            t[pi * 4 + pj] = m[i * 4 + j];
        }
#pragma unroll
    for (int i = 0; i < 16; i++) m[i] = t[i];
}

// Where the builder finds one batch row's parameters.
struct BuildCtx {
    const Member *members;
    const GateDev *gates;
    const int32_t *slot_sym;
    const double *scale, *off;  // this row's scale and offset per slot
    const double *explicit_mats;
    const float *theta;         // this row's symbol values
};

// One build task for one row: symbol resolution eta = scale*theta + offset
// and the fused product / dagger / derivative, all in float64.  D is the
// matrix dimension; fixed at compile time so every array stays in registers.
template <int D> __device__ __forceinline__ void build_task_d(const BuildTask &bt, const BuildCtx &c, double2 *out)
{
    cd acc[16], g[16];
#pragma unroll
    for (int i = 0; i < 16; i++) acc[i] = C(0, 0);
#pragma unroll
    for (int i = 0; i < D; i++) acc[i * D + i] = C(1, 0);
    for (int mi = 0; mi < bt.mem_count; mi++) {
        const Member mem = c.members[bt.mem_begin + mi];
        const GateDev gd = c.gates[mem.gate];
        double eta[2] = {0, 0};
        for (int j = 0; j < gd.np; j++) {
            const int slot = gd.slot0 + j;
            const int sy = c.slot_sym[slot];
            eta[j] = sy >= 0 ? c.scale[slot] * (double)c.theta[sy] + c.off[slot] : c.off[slot];
        }
        const double *ex = gd.explicit_ >= 0 ? c.explicit_mats + 32 * gd.explicit_ : nullptr;
#pragma unroll
        for (int i = 0; i < 16; i++) g[i] = C(0, 0);
        const int gdim = bt.kind == BT_DERIV ? gate_deriv_dev(gd.op, eta, bt.which, mem.form, g)
                                             : gate_matrix_dev(gd.op, eta, ex, mem.form, g);
        if (gdim != D) continue;  // the planner never mixes dimensions
        if (D == 4 && mem.swapped) swap_qubits4(g);
        if (bt.kind == BT_DAGGER) {
#pragma unroll
            for (int i = 0; i < D; i++)
#pragma unroll
                for (int j = 0; j < D; j++) acc[i * D + j] = C(g[j * D + i].x, -g[j * D + i].y);
        } else if (bt.kind == BT_DERIV) {
#pragma unroll
            for (int i = 0; i < D * D; i++) acc[i] = g[i];
        } else {
            cd t[16];
#pragma unroll
            for (int i = 0; i < D; i++)
#pragma unroll
                for (int j = 0; j < D; j++) {
                    cd sacc = C(0, 0);
#pragma unroll
                    for (int k = 0; k < D; k++) sacc = cdadd(sacc, cdmul(g[i * D + k], acc[k * D + j]));
                    t[i * D + j] = sacc;
                }
#pragma unroll
            for (int i = 0; i < D * D; i++) acc[i] = t[i];
        }
    }
    if (bt.diag == 4) {
        // excitation preserving: |00> phase, the (|01>, |10>) block, |11> phase
        const int ix[6] = {0, 5, 6, 9, 10, 15};
#pragma unroll
        for (int i = 0; i < 6; i++) out[i] = make_double2(acc[ix[i]].x, acc[ix[i]].y);
    } else if (bt.diag >= 2) {
        // a I + b P: a from entry (0,0), b from entry (0,3) (P_03 = 1 for XX, -1 for YY)
        const double sg = bt.diag == 3 ? -1.0 : 1.0;
        out[0] = make_double2(acc[0].x, acc[0].y);
        out[1] = make_double2(sg * acc[D - 1].x, sg * acc[D - 1].y);
    } else if (bt.diag) {
#pragma unroll
        for (int i = 0; i < D; i++) out[i] = make_double2(acc[i * D + i].x, acc[i * D + i].y);
    } else {
#pragma unroll
        for (int i = 0; i < D * D; i++) out[i] = make_double2(acc[i].x, acc[i].y);
    }
}

__device__ __forceinline__ void build_task(const BuildTask &bt, const BuildCtx &c, double2 *out)
{
    if (bt.dim == 2) build_task_d<2>(bt, c, out);
    else build_task_d<4>(bt, c, out);
}

// --------------------------------------------------- matrix build kernel
// One thread per (row, task); the result goes to the row's matrix block.
__global__ __launch_bounds__(256) void k_build_mats(BuildArgs a)
{
    const int row = blockIdx.y;
    const int ti = blockIdx.x * blockDim.x + threadIdx.x + a.task_begin;
    if (ti >= a.task_end) return;
    const BuildTask bt = a.tasks[ti];
    const int b = cget(a.rows, row);
    BuildCtx c{a.members, a.gates, a.slot_sym,
               a.slot_scale + (a.uniform ? 0 : (int64_t)row * a.n_slots),
               a.slot_off + (a.uniform ? 0 : (int64_t)row * a.n_slots), a.explicit_mats,
               a.theta + (int64_t)b * a.S};
    build_task(bt, c, a.mats + (int64_t)row * a.mat_stride + bt.out);
}

// ------------------------------------------------------------ tile access
struct TileCtx {
    const uint64_t *hi_off;  // LDS table: global offset of each high-bit combination
    uint32_t lowmask;
    int c;                   // contiguous low bits
};

__device__ __forceinline__ uint64_t tile_index(const TileCtx &tc, uint64_t fb, uint32_t l)
{
    return fb | (l & tc.lowmask) | tc.hi_off[l >> tc.c];
}

// Copy a tile between HBM and LDS, two amplitudes per 16-byte access when
// c >= 1.  Each thread issues a batch of kCopyBatch global accesses before it
// touches LDS, so that a wavefront keeps that many requests in flight instead
// of waiting for every load before the next one is issued.
constexpr int kCopyBatch = 16;
// The per-thread index of a copy is recomputed at every call: the empty asm
// keeps the compiler from hoisting the copies' address arithmetic out of the
// tile loop, where it would stay live across the register-heavy stages.
__device__ __forceinline__ int copy_lane0()
{
    int l = 2 * (int)threadIdx.x;
    asm volatile("" : "+v"(l));
    return l;
}

template <bool kLoad, int kBatch = kCopyBatch>
__device__ __forceinline__ void tile_copy(const TileCtx &tc, float2 *lds, float2 *row, uint64_t fb, int T)
{
    if (tc.c >= 1) {
        const int step = 2 * blockDim.x;
        for (int l0 = copy_lane0(); l0 < T; l0 += kBatch * step) {
            float4 v[kBatch];
            if (kLoad) {
#pragma unroll
                for (int k = 0; k < kBatch; k++) {
                    const int l = l0 + k * step;
                    if (l < T) v[k] = *reinterpret_cast<const float4 *>(row + tile_index(tc, fb, l));
                }
#pragma unroll
                for (int k = 0; k < kBatch; k++) {
                    const int l = l0 + k * step;
                    if (l < T) {
                        lds[sw(l)] = make_float2(v[k].x, v[k].y);
                        lds[sw(l + 1)] = make_float2(v[k].z, v[k].w);
                    }
                }
            } else {
#pragma unroll
                for (int k = 0; k < kBatch; k++) {
                    const int l = l0 + k * step;
                    if (l < T) {
                        const float2 u0 = lds[sw(l)], u1 = lds[sw(l + 1)];
                        v[k] = make_float4(u0.x, u0.y, u1.x, u1.y);
                    }
                }
#pragma unroll
                for (int k = 0; k < kBatch; k++) {
                    const int l = l0 + k * step;
                    if (l < T) *reinterpret_cast<float4 *>(row + tile_index(tc, fb, l)) = v[k];
                }
            }
        }
    } else {
        for (int l = threadIdx.x; l < T; l += blockDim.x) {
            if (kLoad) lds[sw(l)] = row[tile_index(tc, fb, l)];
            else row[tile_index(tc, fb, l)] = lds[sw(l)];
        }
    }
}

__device__ void build_hi_off(const TileGeom &g, uint64_t *hi_off)
{
    for (int j = threadIdx.x; j < (1 << g.h); j += blockDim.x) {
        uint64_t o = 0;
        for (int k = 0; k < g.h; k++)
            if ((j >> k) & 1) o |= 1ull << g.hb[k];
        hi_off[j] = o;
    }
}

__device__ __forceinline__ int bit_of(uint8_t loc, uint8_t pos, uint32_t l, uint64_t fb)
{
    return loc != kFixed ? (int)((l >> loc) & 1) : (int)((fb >> pos) & 1);
}

// ------------------------------------------------------ forward tile ops
// Diagonal entry index of local element l: 2*bit(q0) + bit(q1) for K_D2,
// bit(q0) for K_D1, each bit taken from the tile index or the fixed bits.
__device__ __forceinline__ int diag_index(const PassOp &op, uint32_t l, uint64_t fb)
{
    int idx = bit_of(op.l0, op.p0, l, fb);
    if (op.kind == K_D2) idx = 2 * idx + bit_of(op.l1, op.p1, l, fb);
    return idx;
}

// (a I + b P) on the quad (v00, v01, v10, v11); P = XX (sg = 1) or YY
// (sg = -1): P couples 00 with 11 (sign sg) and 01 with 10 (sign +1)
struct Quad {
    double2 v00, v01, v10, v11;
};
__device__ __forceinline__ Quad p2_apply(double2 a, double2 b, double sg, const Quad &v)
{
    const double2 bs = make_double2(sg * b.x, sg * b.y);
    Quad o;
    o.v00 = zadd(zmul(a, v.v00), zmul(bs, v.v11));
    o.v11 = zadd(zmul(a, v.v11), zmul(bs, v.v00));
    o.v01 = zadd(zmul(a, v.v01), zmul(b, v.v10));
    o.v10 = zadd(zmul(a, v.v10), zmul(b, v.v01));
    return o;
}

// Matrix entries seen by the register ops: a pointer into LDS, or an SMat,
// which reads a row's matrix block in HBM through the scalar cache (uniform
// indices land in scalar registers and feed the FMAs directly).
struct SMat {
    const __attribute__((address_space(4))) double *p;
    __device__ __forceinline__ double2 operator[](int i) const { return make_double2(p[2 * i], p[2 * i + 1]); }
    __device__ __forceinline__ SMat operator+(int i) const { return SMat{p + 2 * i}; }
};
__device__ __forceinline__ SMat smat(const double2 *block)
{
    return SMat{(const __attribute__((address_space(4))) double *)block};
}

// ------------------------------------------------------- register stages
// A stage's ops run on the 2^R amplitudes one thread holds in registers (in
// fp64); register index k has bit j set when tile bit stage.bits[j] is set.
// An op bit outside the stage comes from the item's base index or the fixed
// bits of the tile.

// Register-level ops.  Every variant is a template on the register bits it
// touches, so the element pattern is fixed at compile time (no selects).

// dense 2x2 on register bit J
template <int R, int J, class MT> __device__ __forceinline__ void rm1(double2 *a, MT m)
{
    const double2 m00 = m[0], m01 = m[1], m10 = m[2], m11 = m[3];
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if ((k >> J) & 1) continue;
        const int kk = k | (1 << J);
        const double2 x = a[k], y = a[kk];
        a[k] = zmul2(m00, x, m01, y);
        a[kk] = zmul2(m10, x, m11, y);
    }
}
// sum of Re(conj(f) (dm a)) over the pairs of rm1
template <int R, int J, class MT> __device__ __forceinline__ double rm1_dot(const double2 *a, const double2 *f, MT dm)
{
    const double2 m00 = dm[0], m01 = dm[1], m10 = dm[2], m11 = dm[3];
    double s = 0;
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if ((k >> J) & 1) continue;
        const int kk = k | (1 << J);
        s += zdotr(f[k], zmul2(m00, a[k], m01, a[kk])) + zdotr(f[kk], zmul2(m10, a[k], m11, a[kk]));
    }
    return s;
}
// dense 2x2 on register bit J where register bit C is 1 (controlled gates)
template <int R, int J, int C, class MT> __device__ __forceinline__ void rm1c(double2 *a, MT m)
{
    const double2 m00 = m[0], m01 = m[1], m10 = m[2], m11 = m[3];
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if (((k >> J) & 1) || !((k >> C) & 1)) continue;
        const int kk = k | (1 << J);
        const double2 x = a[k], y = a[kk];
        a[k] = zmul2(m00, x, m01, y);
        a[kk] = zmul2(m10, x, m11, y);
    }
}
template <int R, int J, int C, class MT>
__device__ __forceinline__ double rm1c_dot(const double2 *a, const double2 *f, MT dm)
{
    const double2 m00 = dm[0], m01 = dm[1], m10 = dm[2], m11 = dm[3];
    double s = 0;
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if (((k >> J) & 1) || !((k >> C) & 1)) continue;
        const int kk = k | (1 << J);
        s += zdotr(f[k], zmul2(m00, a[k], m01, a[kk])) + zdotr(f[kk], zmul2(m10, a[k], m11, a[kk]));
    }
    return s;
}
// diagonal (e0, e1) on register bit J
template <int R, int J> __device__ __forceinline__ void rd1(double2 *a, double2 e0, double2 e1)
{
#pragma unroll
    for (int k = 0; k < (1 << R); k++) a[k] = zmul(((k >> J) & 1) ? e1 : e0, a[k]);
}
template <int R, int J> __device__ __forceinline__ double rd1_dot(const double2 *a, const double2 *f, double2 e0, double2 e1)
{
    double s = 0;
#pragma unroll
    for (int k = 0; k < (1 << R); k++) s += zdotr(f[k], zmul(((k >> J) & 1) ? e1 : e0, a[k]));
    return s;
}
// diagonal on register bits (LO, HI), entry index 2*bit(LO) + bit(HI)
template <int R, int LO, int HI>
__device__ __forceinline__ void rd2(double2 *a, double2 e0, double2 e1, double2 e2, double2 e3)
{
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        const int idx = 2 * ((k >> LO) & 1) + ((k >> HI) & 1);
        a[k] = zmul(idx == 0 ? e0 : idx == 1 ? e1 : idx == 2 ? e2 : e3, a[k]);
    }
}
template <int R, int LO, int HI>
__device__ __forceinline__ double rd2_dot(const double2 *a, const double2 *f, double2 e0, double2 e1, double2 e2, double2 e3)
{
    double s = 0;
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        const int idx = 2 * ((k >> LO) & 1) + ((k >> HI) & 1);
        s += zdotr(f[k], zmul(idx == 0 ? e0 : idx == 1 ? e1 : idx == 2 ? e2 : e3, a[k]));
    }
    return s;
}
template <int R> __device__ __forceinline__ void rscale(double2 *a, double2 e)
{
#pragma unroll
    for (int k = 0; k < (1 << R); k++) a[k] = zmul(e, a[k]);
}
template <int R> __device__ __forceinline__ double rscale_dot(const double2 *a, const double2 *f, double2 e)
{
    double s = 0;
#pragma unroll
    for (int k = 0; k < (1 << R); k++) s += zdotr(f[k], zmul(e, a[k]));
    return s;
}

// dense 4x4 on register bits (LO = the op's first qubit, HI = its second):
// local index 2*bit(q0) + bit(q1) = 2*bit(LO) + bit(HI)
template <int R, int LO, int HI, class MT> __device__ __forceinline__ void rm2(double2 *a, MT m)
{
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if (((k >> LO) & 1) || ((k >> HI) & 1)) continue;
        const int k10 = k | (1 << LO), k01 = k | (1 << HI), k11 = k10 | k01;
        const double2 v00 = a[k], v01 = a[k01], v10 = a[k10], v11 = a[k11];
        a[k] = zadd(zmul2(m[0], v00, m[1], v01), zmul2(m[2], v10, m[3], v11));
        a[k01] = zadd(zmul2(m[4], v00, m[5], v01), zmul2(m[6], v10, m[7], v11));
        a[k10] = zadd(zmul2(m[8], v00, m[9], v01), zmul2(m[10], v10, m[11], v11));
        a[k11] = zadd(zmul2(m[12], v00, m[13], v01), zmul2(m[14], v10, m[15], v11));
    }
}
template <int R, int LO, int HI, class MT> __device__ __forceinline__ double rm2_dot(const double2 *a, const double2 *f, MT m)
{
    double s = 0;
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if (((k >> LO) & 1) || ((k >> HI) & 1)) continue;
        const int k10 = k | (1 << LO), k01 = k | (1 << HI), k11 = k10 | k01;
        const double2 v00 = a[k], v01 = a[k01], v10 = a[k10], v11 = a[k11];
        s += zdotr(f[k], zadd(zmul2(m[0], v00, m[1], v01), zmul2(m[2], v10, m[3], v11)));
        s += zdotr(f[k01], zadd(zmul2(m[4], v00, m[5], v01), zmul2(m[6], v10, m[7], v11)));
        s += zdotr(f[k10], zadd(zmul2(m[8], v00, m[9], v01), zmul2(m[10], v10, m[11], v11)));
        s += zdotr(f[k11], zadd(zmul2(m[12], v00, m[13], v01), zmul2(m[14], v10, m[15], v11)));
    }
    return s;
}
// excitation preserving on (LO = q0, HI = q1): m = {p00, b00, b01, b10, b11, p11};
// out01 = b00 v01 + b01 v10, out10 = b10 v01 + b11 v10
template <int R, int LO, int HI, class MT> __device__ __forceinline__ void rf2(double2 *a, MT m)
{
    const double2 p00 = m[0], b00 = m[1], b01 = m[2], b10 = m[3], b11 = m[4], p11 = m[5];
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if (((k >> LO) & 1) || ((k >> HI) & 1)) continue;
        const int k10 = k | (1 << LO), k01 = k | (1 << HI), k11 = k10 | k01;
        const double2 v01 = a[k01], v10 = a[k10];
        a[k] = zmul(p00, a[k]);
        a[k01] = zmul2(b00, v01, b01, v10);
        a[k10] = zmul2(b10, v01, b11, v10);
        a[k11] = zmul(p11, a[k11]);
    }
}
template <int R, int LO, int HI, class MT> __device__ __forceinline__ double rf2_dot(const double2 *a, const double2 *f, MT m)
{
    const double2 p00 = m[0], b00 = m[1], b01 = m[2], b10 = m[3], b11 = m[4], p11 = m[5];
    double s = 0;
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if (((k >> LO) & 1) || ((k >> HI) & 1)) continue;
        const int k10 = k | (1 << LO), k01 = k | (1 << HI), k11 = k10 | k01;
        s += zdotr(f[k], zmul(p00, a[k])) + zdotr(f[k11], zmul(p11, a[k11]));
        s += zdotr(f[k01], zmul2(b00, a[k01], b01, a[k10])) + zdotr(f[k10], zmul2(b10, a[k01], b11, a[k10]));
    }
    return s;
}

// a I + b P on register bits (LO, HI); P = XX (sg = 1) or YY (sg = -1), symmetric in the two qubits
template <int R, int LO, int HI> __device__ __forceinline__ void rp2(double2 *a, double2 ca, double2 cb, double sg)
{
    const double2 bs = make_double2(sg * cb.x, sg * cb.y);
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if (((k >> LO) & 1) || ((k >> HI) & 1)) continue;
        const int kL = k | (1 << LO), kH = k | (1 << HI), k11 = kL | kH;
        const double2 v00 = a[k], vL = a[kL], vH = a[kH], v11 = a[k11];
        a[k] = zadd(zmul(ca, v00), zmul(bs, v11));
        a[k11] = zadd(zmul(ca, v11), zmul(bs, v00));
        a[kL] = zadd(zmul(ca, vL), zmul(cb, vH));
        a[kH] = zadd(zmul(ca, vH), zmul(cb, vL));
    }
}
template <int R, int LO, int HI> __device__ __forceinline__ double rp2_dot(const double2 *a, const double2 *f, double2 ca, double2 cb, double sg)
{
    const double2 bs = make_double2(sg * cb.x, sg * cb.y);
    double s = 0;
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if (((k >> LO) & 1) || ((k >> HI) & 1)) continue;
        const int kL = k | (1 << LO), kH = k | (1 << HI), k11 = kL | kH;
        s += zdotr(f[k], zadd(zmul(ca, a[k]), zmul(bs, a[k11])));
        s += zdotr(f[k11], zadd(zmul(ca, a[k11]), zmul(bs, a[k])));
        s += zdotr(f[kL], zadd(zmul(ca, a[kL]), zmul(cb, a[kH])));
        s += zdotr(f[kH], zadd(zmul(ca, a[kH]), zmul(cb, a[kL])));
    }
    return s;
}

// Runtime register bit(s) -> template instantiation, written out as switches
// (no lambdas: the register arrays must stay in registers).  Each switch
// covers exactly the valid cases of its R, the last one as `default`: a
// switch with a path that leaves the registers untouched makes the compiler
// copy the whole register array on every op.
#define TQ_C1(J_, CALL) { constexpr int j_ = J_; CALL; } break;
#define TQ_BIT_SWITCH(R, J, CALL)                                                                                   \
    if constexpr (R == 1) {                                                                                         \
        constexpr int j_ = 0; CALL;                                                                                 \
    } else if constexpr (R == 2) {                                                                                  \
        switch (J) { case 0: TQ_C1(0, CALL) default: TQ_C1(1, CALL) }                                              \
    } else if constexpr (R == 3) {                                                                                  \
        switch (J) { case 0: TQ_C1(0, CALL) case 1: TQ_C1(1, CALL) default: TQ_C1(2, CALL) }                       \
    } else if constexpr (R == 4) {                                                                                  \
        switch (J) { case 0: TQ_C1(0, CALL) case 1: TQ_C1(1, CALL) case 2: TQ_C1(2, CALL) default: TQ_C1(3, CALL) } \
    }
#define TQ_C2(L_, H_, CALL) { constexpr int lo_ = L_, hi_ = H_; CALL; } break;
#define TQ_PAIR_SWITCH(R, LO, HI, CALL)                                                                             \
    if constexpr (R == 2) {                                                                                         \
        constexpr int lo_ = 0, hi_ = 1; CALL;                                                                       \
    } else if constexpr (R == 3) {                                                                                  \
        switch ((LO) * 4 + (HI)) { case 1: TQ_C2(0, 1, CALL) case 2: TQ_C2(0, 2, CALL) default: TQ_C2(1, 2, CALL) } \
    } else if constexpr (R == 4) {                                                                                  \
        switch ((LO) * 4 + (HI)) {                                                                                  \
        case 1: TQ_C2(0, 1, CALL) case 2: TQ_C2(0, 2, CALL) case 3: TQ_C2(0, 3, CALL)                               \
        case 6: TQ_C2(1, 2, CALL) case 7: TQ_C2(1, 3, CALL) default: TQ_C2(2, 3, CALL)                              \
        }                                                                                                           \
    }
#define TQ_CO(J_, C_, CALL) { constexpr int j_ = J_, c_ = C_; CALL; } break;
#define TQ_ORDERED_SWITCH(R, J, C, CALL)                                                                            \
    if constexpr (R == 2) {                                                                                         \
        switch ((J) * 4 + (C)) { case 1: TQ_CO(0, 1, CALL) default: TQ_CO(1, 0, CALL) }                            \
    } else if constexpr (R == 3) {                                                                                  \
        switch ((J) * 4 + (C)) {                                                                                    \
        case 1: TQ_CO(0, 1, CALL) case 2: TQ_CO(0, 2, CALL) case 4: TQ_CO(1, 0, CALL)                               \
        case 6: TQ_CO(1, 2, CALL) case 8: TQ_CO(2, 0, CALL) default: TQ_CO(2, 1, CALL)                              \
        }                                                                                                           \
    } else if constexpr (R == 4) {                                                                                  \
        switch ((J) * 4 + (C)) {                                                                                    \
        case 1: TQ_CO(0, 1, CALL) case 2: TQ_CO(0, 2, CALL) case 3: TQ_CO(0, 3, CALL)                               \
        case 4: TQ_CO(1, 0, CALL) case 6: TQ_CO(1, 2, CALL) case 7: TQ_CO(1, 3, CALL)                               \
        case 8: TQ_CO(2, 0, CALL) case 9: TQ_CO(2, 1, CALL) case 11: TQ_CO(2, 3, CALL)                              \
        case 12: TQ_CO(3, 0, CALL) case 13: TQ_CO(3, 1, CALL) default: TQ_CO(3, 2, CALL)                            \
        }                                                                                                           \
    }

// How a diagonal op acts on a stage item: both bits in registers, one bit
// (the other one's value fixed for the item), or none (one scalar).
struct DiagPlan {
    int mode;     // 0: scalar, 1: one register bit, 2: two register bits
    int j0, j1;   // register bits (mode 1: j0; mode 2: j0 < j1)
    int e[4];     // entry indices, ordered by the register bits' pattern
};
__device__ __forceinline__ DiagPlan diag_plan(const PassOp &op, uint32_t base, uint64_t fb)
{
    DiagPlan d{};
    if (op.kind == K_D1) {
        if (op.s0 != kFixed) {
            d.mode = 1;
            d.j0 = op.s0;
            d.e[0] = 0;
            d.e[1] = 1;
        } else {
            d.mode = 0;
            d.e[0] = bit_of(op.l0, op.p0, base, fb);
        }
        return d;
    }
    const bool r0 = op.s0 != kFixed, r1 = op.s1 != kFixed;
    if (r0 && r1) {
        d.mode = 2;
        d.j0 = min(op.s0, op.s1);
        d.j1 = max(op.s0, op.s1);
        // idx = 2*bit(q0) + bit(q1); pattern index = 2*bit(j0) + bit(j1)
        const bool q0lo = op.s0 < op.s1;
        d.e[0] = 0;
        d.e[1] = q0lo ? 1 : 2;
        d.e[2] = q0lo ? 2 : 1;
        d.e[3] = 3;
    } else if (r0) {
        d.mode = 1;
        d.j0 = op.s0;
        const int v = bit_of(op.l1, op.p1, base, fb);
        d.e[0] = v;
        d.e[1] = 2 + v;
    } else if (r1) {
        d.mode = 1;
        d.j0 = op.s1;
        const int v = bit_of(op.l0, op.p0, base, fb);
        d.e[0] = 2 * v;
        d.e[1] = 2 * v + 1;
    } else {
        d.mode = 0;
        d.e[0] = 2 * bit_of(op.l0, op.p0, base, fb) + bit_of(op.l1, op.p1, base, fb);
    }
    return d;
}

template <int R, class MT> __device__ __forceinline__ void reg_diag(const DiagPlan &d, MT m, double2 *a)
{
    if (d.mode == 0) {
        rscale<R>(a, m[d.e[0]]);
    } else if (d.mode == 1) {
        const double2 e0 = m[d.e[0]], e1 = m[d.e[1]];
        TQ_BIT_SWITCH(R, d.j0, (rd1<R, j_>(a, e0, e1)))
    } else {
        const double2 e0 = m[d.e[0]], e1 = m[d.e[1]], e2 = m[d.e[2]], e3 = m[d.e[3]];
        TQ_PAIR_SWITCH(R, d.j0, d.j1, (rd2<R, lo_, hi_>(a, e0, e1, e2, e3)))
    }
}
template <int R, class MT> __device__ __forceinline__ double reg_diag_dot(const DiagPlan &d, MT m, const double2 *a, const double2 *f)
{
    double s = 0;
    if (d.mode == 0) {
        s = rscale_dot<R>(a, f, m[d.e[0]]);
    } else if (d.mode == 1) {
        const double2 e0 = m[d.e[0]], e1 = m[d.e[1]];
        TQ_BIT_SWITCH(R, d.j0, (s = rd1_dot<R, j_>(a, f, e0, e1)))
    } else {
        const double2 e0 = m[d.e[0]], e1 = m[d.e[1]], e2 = m[d.e[2]], e3 = m[d.e[3]];
        TQ_PAIR_SWITCH(R, d.j0, d.j1, (s = rd2_dot<R, lo_, hi_>(a, f, e0, e1, e2, e3)))
    }
    return s;
}

// A K_M1 op whose control bit lies outside the stage acts on an item only
// when that bit (from the item's base index or the tile's fixed bits) is 1.
// The matrix is selected per lane -- the op's or the identity -- so that
// every path writes the registers.
struct Mat2 {
    double2 e[4];
    __device__ __forceinline__ double2 operator[](int i) const { return e[i]; }
};
template <class MT> __device__ __forceinline__ Mat2 ctrl_sel(MT m, bool on)
{
    const double2 one = make_double2(1.0, 0.0), zero = make_double2(0.0, 0.0);
    Mat2 r;
    r.e[0] = on ? m[0] : one;
    r.e[1] = on ? m[1] : zero;
    r.e[2] = on ? m[2] : zero;
    r.e[3] = on ? m[3] : one;
    return r;
}
__device__ __forceinline__ bool ctrl_on(const PassOp &op, uint32_t base, uint64_t fb)
{
    return bit_of(op.l1, op.p1, base, fb) == op.cval;
}

// forward op on registers
template <int R, class MT> __device__ __forceinline__ void reg_op(const PassOp &op, MT m, double2 *a, uint32_t base, uint64_t fb)
{
    switch (op.kind) {
    case K_M1: {
        if (!op.ctrl) {
            TQ_BIT_SWITCH(R, op.s0, (rm1<R, j_>(a, m)))
        } else if (op.s1 != kFixed) {
            TQ_ORDERED_SWITCH(R, op.s0, op.s1, (rm1c<R, j_, c_>(a, m)))
        } else {
            const Mat2 ms = ctrl_sel(m, ctrl_on(op, base, fb));
            TQ_BIT_SWITCH(R, op.s0, (rm1<R, j_>(a, ms)))
        }
        return;
    }
    case K_M2: TQ_PAIR_SWITCH(R, op.s0, op.s1, (rm2<R, lo_, hi_>(a, m))) return;
    case K_F2: TQ_PAIR_SWITCH(R, op.s0, op.s1, (rf2<R, lo_, hi_>(a, m))) return;
    case K_P2: {
        const double sg = op.ptype == 2 ? -1.0 : 1.0;
        const double2 ca = m[0], cb = m[1];
        TQ_PAIR_SWITCH(R, min(op.s0, op.s1), max(op.s0, op.s1), (rp2<R, lo_, hi_>(a, ca, cb, sg)))
        return;
    }
    default: reg_diag<R>(diag_plan(op, base, fb), m, a); return;
    }
}

// reverse op on registers: a <- W^dagger a (m = W^dagger); g_j += sum Re(conj(f) dW_j a);
// f <- W^dagger f
template <int R, class MT>
__device__ __forceinline__ void reg_rev_op(const PassOp &op, MT m, MT d0, MT d1,
                                           double2 *a, double2 *f, uint32_t base, uint64_t fb, double &g0, double &g1)
{
    switch (op.kind) {
    case K_M1: {
        if (!op.ctrl) {
            TQ_BIT_SWITCH(R, op.s0, ({
                rm1<R, j_>(a, m);
                if (op.ngrad > 0) g0 += rm1_dot<R, j_>(a, f, d0);
                if (op.ngrad > 1) g1 += rm1_dot<R, j_>(a, f, d1);
                rm1<R, j_>(f, m);
            }))
        } else if (op.s1 != kFixed) {
            TQ_ORDERED_SWITCH(R, op.s0, op.s1, ({
                rm1c<R, j_, c_>(a, m);
                if (op.ngrad > 0) g0 += rm1c_dot<R, j_, c_>(a, f, d0);
                if (op.ngrad > 1) g1 += rm1c_dot<R, j_, c_>(a, f, d1);
                rm1c<R, j_, c_>(f, m);
            }))
        } else {
            // an item whose control is off sees the identity and a zero derivative
            const bool on = ctrl_on(op, base, fb);
            const Mat2 ms = ctrl_sel(m, on);
            TQ_BIT_SWITCH(R, op.s0, ({
                rm1<R, j_>(a, ms);
                if (op.ngrad > 0) g0 += on ? rm1_dot<R, j_>(a, f, d0) : 0.0;
                if (op.ngrad > 1) g1 += on ? rm1_dot<R, j_>(a, f, d1) : 0.0;
                rm1<R, j_>(f, ms);
            }))
        }
        return;
    }
    case K_M2:
        // dense two-qubit ops only occur in stages of at most kRevDense2Bits
        // register bits (planner): wider instances are not compiled
        if constexpr (R <= kRevDense2Bits) {
            TQ_PAIR_SWITCH(R, op.s0, op.s1, ({
                rm2<R, lo_, hi_>(a, m);
                if (op.ngrad > 0) g0 += rm2_dot<R, lo_, hi_>(a, f, d0);
                if (op.ngrad > 1) g1 += rm2_dot<R, lo_, hi_>(a, f, d1);
                rm2<R, lo_, hi_>(f, m);
            }))
        }
        return;
    case K_F2:
        if constexpr (R <= kRevDense2Bits) {
            TQ_PAIR_SWITCH(R, op.s0, op.s1, ({
                rf2<R, lo_, hi_>(a, m);
                if (op.ngrad > 0) g0 += rf2_dot<R, lo_, hi_>(a, f, d0);
                if (op.ngrad > 1) g1 += rf2_dot<R, lo_, hi_>(a, f, d1);
                rf2<R, lo_, hi_>(f, m);
            }))
        }
        return;
    case K_P2: {
        const double sg = op.ptype == 2 ? -1.0 : 1.0;
        const double2 ca = m[0], cb = m[1];
        TQ_PAIR_SWITCH(R, min(op.s0, op.s1), max(op.s0, op.s1), ({
            rp2<R, lo_, hi_>(a, ca, cb, sg);
            if (op.ngrad > 0) g0 += rp2_dot<R, lo_, hi_>(a, f, d0[0], d0[1], sg);
            rp2<R, lo_, hi_>(f, ca, cb, sg);
        }))
        return;
    }
    default: {
        const DiagPlan d = diag_plan(op, base, fb);
        reg_diag<R>(d, m, a);
        if (op.ngrad > 0) g0 += reg_diag_dot<R>(d, d0, a, f);
        if (op.ngrad > 1) g1 += reg_diag_dot<R>(d, d1, a, f);
        reg_diag<R>(d, m, f);
        return;
    }
    }
}

// LDS offsets of a stage's register elements
template <int R> __device__ __forceinline__ void stage_offsets(const Stage &st, uint32_t *off)
{
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        uint32_t o = 0;
#pragma unroll
        for (int j = 0; j < R; j++)
            if ((k >> j) & 1) o |= 1u << st.bits[j];
        off[k] = o;
    }
}

template <int R> __device__ __forceinline__ uint32_t stage_base(const Stage &st, uint32_t item)
{
    uint32_t base = item;
#pragma unroll
    for (int j = 0; j < R; j++) base = ins0(base, st.bits[j]);
    return base;
}

// One forward stage over a tile of 2^t amplitudes in LDS.  M holds the
// matrices from row-block offset mbase on.
// Dense stage: a <- S a with the 2^R x 2^R stage matrix S (row major),
// read through the scalar cache.
template <int R> __device__ __forceinline__ void rdense(double2 *a, SMat S)
{
    constexpr int N = 1 << R;
    double2 b[N];
#pragma unroll
    for (int k = 0; k < N; k++) {
        double re = 0.0, im = 0.0;
#pragma unroll
        for (int j = 0; j < N; j++) {
            const double2 m = S[k * N + j];
            re = fma(m.x, a[j].x, fma(-m.y, a[j].y, re));
            im = fma(m.x, a[j].y, fma(m.y, a[j].x, im));
        }
        b[k] = make_double2(re, im);
    }
#pragma unroll
    for (int k = 0; k < N; k++) a[k] = b[k];
}

template <int R, class MT>
__device__ __forceinline__ void run_stage(const Stage &st, const PassOp *ops, MT M, int mbase, SMat G, float2 *lds, int t,
                                          uint64_t fb, int tid, int nt)
{
    // sw() is linear over xor and base, off[k] have disjoint bits, so the
    // swizzled address of base | off[k] is sw(base) ^ sw(off[k])
    uint32_t off[1 << R];
    stage_offsets<R>(st, off);
#pragma unroll
    for (int k = 0; k < (1 << R); k++) off[k] = sw(off[k]);
    const uint32_t nitems = 1u << (t - R);
    for (uint32_t item = tid; item < nitems; item += nt) {
        const uint32_t base = stage_base<R>(st, item), sb = sw(base);
        double2 a[1 << R];
#pragma unroll
        for (int k = 0; k < (1 << R); k++) a[k] = up2(lds[sb ^ off[k]]);
        if (st.dense) {
            rdense<R>(a, G + st.mat);
        } else {
            for (int oi = st.op_begin; oi < st.op_end; oi++) {
                const PassOp op = cget(ops, oi);
                reg_op<R>(op, M + (op.mat - mbase), a, base, fb);
            }
        }
#pragma unroll
        for (int k = 0; k < (1 << R); k++) lds[sb ^ off[k]] = down2(a[k]);
    }
}

// tid / nt: this thread's index among the nt threads that share the tile;
// G: the row's matrix block in HBM (dense stage matrices)
template <class MT>
__device__ __forceinline__ void run_stage_any(const Stage &st, const PassOp *ops, MT M, int mbase, SMat G, float2 *lds, int t,
                                              uint64_t fb, int tid, int nt)
{
    switch (st.r) {
    case 4:
        if constexpr (kStageBitsFwd >= 4) run_stage<4>(st, ops, M, mbase, G, lds, t, fb, tid, nt);
        break;
    case 3: run_stage<3>(st, ops, M, mbase, G, lds, t, fb, tid, nt); break;
    case 2: run_stage<2>(st, ops, M, mbase, G, lds, t, fb, tid, nt); break;
    case 1: run_stage<1>(st, ops, M, mbase, G, lds, t, fb, tid, nt); break;
    default: run_stage<0>(st, ops, M, mbase, G, lds, t, fb, tid, nt); break;
    }
}

// Register accumulators of a stage's gradient parameters, indexed by a
// uniform k < kMaxStageGrads (a branch, so that the array stays in registers).
__device__ __forceinline__ void gadd(double *g, int k, double v)
{
    switch (k) {
    case 0: g[0] += v; break;
    case 1: g[1] += v; break;
    case 2: g[2] += v; break;
    case 3: g[3] += v; break;
    case 4: g[4] += v; break;
    case 5: g[5] += v; break;
    case 6: g[6] += v; break;
    default: g[7] += v; break;
    }
}
__device__ __forceinline__ double gget(const double *g, int k)
{
    switch (k) {
    case 0: return g[0];
    case 1: return g[1];
    case 2: return g[2];
    case 3: return g[3];
    case 4: return g[4];
    case 5: return g[5];
    case 6: return g[6];
    default: return g[7];
    }
}
static_assert(kMaxStageGrads == 8, "gadd/gget cover eight accumulators");

// One reverse stage on the psi and phi tiles.  Each thread sums the
// gradient contributions of its items in registers; after the items, one
// wavefront reduction per gradient parameter adds into
// acc[wave * astride + slot - abase].
template <int R, class MT>
__device__ __forceinline__ void run_rev_stage(const Stage &st, const PassOp *ops, MT M, int mbase, float2 *lp, float2 *lf,
                              int t, uint64_t fb, double *acc, int astride, int abase, int tid, int nt)
{
    uint32_t off[1 << R];
    stage_offsets<R>(st, off);
#pragma unroll
    for (int k = 0; k < (1 << R); k++) off[k] = sw(off[k]);  // see run_stage
    const uint32_t nitems = 1u << (t - R);
    const int wave = tid / 64, lane = tid % 64;
    double gacc[kMaxStageGrads];
#pragma unroll
    for (int j = 0; j < kMaxStageGrads; j++) gacc[j] = 0.0;
    for (uint32_t item = tid; item < nitems; item += nt) {
        const uint32_t base = stage_base<R>(st, item), sb = sw(base);
        double2 a[1 << R], f[1 << R];
#pragma unroll
        for (int k = 0; k < (1 << R); k++) {
            a[k] = up2(lp[sb ^ off[k]]);
            f[k] = up2(lf[sb ^ off[k]]);
        }
        int gk = 0;
        for (int oi = st.op_begin; oi < st.op_end; oi++) {
            const PassOp op = cget(ops, oi);
            const MT m = M + (op.mat - mbase);
            const MT d0 = M + (op.ngrad > 0 ? op.dmat[0] - mbase : 0);
            const MT d1 = M + (op.ngrad > 1 ? op.dmat[1] - mbase : 0);
            double g0 = 0, g1 = 0;
            reg_rev_op<R>(op, m, d0, d1, a, f, base, fb, g0, g1);
            if (op.ngrad > 0) gadd(gacc, gk++, g0);
            if (op.ngrad > 1) gadd(gacc, gk++, g1);
        }
#pragma unroll
        for (int k = 0; k < (1 << R); k++) {
            lp[sb ^ off[k]] = down2(a[k]);
            lf[sb ^ off[k]] = down2(f[k]);
        }
    }
    int gk = 0;
    for (int oi = st.op_begin; oi < st.op_end; oi++) {
        const PassOp op = cget(ops, oi);
        for (int j = 0; j < op.ngrad; j++) {
            const double v = wave_sum(gget(gacc, gk++));
            const int slot = j == 0 ? op.gslot[0] : op.gslot[1];
            if (lane == 0) acc[wave * astride + slot - abase] += v;
        }
    }
}

// kRMax: the widest stage the caller's plans contain (narrower kernels
// compile fewer register variants)
template <int kRMax, class MT>
__device__ __forceinline__ void run_rev_stage_any(const Stage &st, const PassOp *ops, MT M, int mbase, float2 *lp, float2 *lf,
                                  int t, uint64_t fb, double *acc, int astride, int abase, int tid, int nt)
{
    switch (st.r) {
    case 3:
        if constexpr (kRMax >= 3) run_rev_stage<3>(st, ops, M, mbase, lp, lf, t, fb, acc, astride, abase, tid, nt);
        break;
    case 2: run_rev_stage<2>(st, ops, M, mbase, lp, lf, t, fb, acc, astride, abase, tid, nt); break;
    case 1: run_rev_stage<1>(st, ops, M, mbase, lp, lf, t, fb, acc, astride, abase, tid, nt); break;
    default: run_rev_stage<0>(st, ops, M, mbase, lp, lf, t, fb, acc, astride, abase, tid, nt); break;
    }
}

// Dense stage matrices: column j of a stage's matrix is the stage's ops
// applied to the basis vector e_j (the same register ops the op-by-op path
// runs), one thread per column, in fp64.
template <int R> __device__ __forceinline__ void build_stage_r(const Stage &st, const PassOp *ops, const double2 *block,
                                                              double2 *out, int j)
{
    constexpr int N = 1 << R;
    double2 a[N];
#pragma unroll
    for (int k = 0; k < N; k++) a[k] = make_double2(k == j ? 1.0 : 0.0, 0.0);
    for (int oi = st.op_begin; oi < st.op_end; oi++) {
        const PassOp op = cget(ops, oi);
        reg_op<R>(op, block + op.mat, a, 0u, 0ull);
    }
#pragma unroll
    for (int k = 0; k < N; k++) out[k * N + j] = a[k];
}

__global__ __launch_bounds__(64) void k_build_stage(StageBuildArgs a)
{
    const int si = blockIdx.x, row = blockIdx.y, j = threadIdx.x;
    const Stage st = cget(a.stages, cget(a.list, si));
    if (j >= (1 << st.r)) return;
    double2 *block = a.mats + (int64_t)row * a.mat_stride;
    double2 *out = block + st.mat;
    switch (st.r) {
    case 4:
        if constexpr (kStageBitsFwd >= 4) build_stage_r<4>(st, a.ops, block, out, j);
        break;
    case 3: build_stage_r<3>(st, a.ops, block, out, j); break;
    case 2: build_stage_r<2>(st, a.ops, block, out, j); break;
    default: build_stage_r<1>(st, a.ops, block, out, j); break;
    }
}

// Stage the matrices [begin, end) of a row block into LDS.
__device__ __forceinline__ void stage_mats(double2 *dst, const double2 *row_block, int begin, int end)
{
    for (int i = begin + (int)threadIdx.x; i < end; i += blockDim.x) dst[i - begin] = row_block[i];
}

// ------------------------------------------------------- forward pass
__global__ __launch_bounds__(256) void k_pass(PassArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const TileGeom &g = a.g;
    const int t = g.t;
    const int T = 1 << t;
    float2 *lds = reinterpret_cast<float2 *>(smem);
    uint64_t *hi_off = reinterpret_cast<uint64_t *>(smem + sizeof(float2) * T);
    double2 *lm = reinterpret_cast<double2 *>(hi_off + (1 << g.h));  // the pass's matrices
    double2 *p1 = lm + (a.mat_end - a.mat_begin);
    const int a1 = t / 2;
    double2 *p2 = p1 + (1 << a1);

    const int row = blockIdx.x / a.wg_per_row, w = blockIdx.x % a.wg_per_row;
    const int b = cget(a.rows, row);
    float2 *st = a.state + (int64_t)b * a.row_stride;
    build_hi_off(g, hi_off);
    stage_mats(lm, a.mats + (int64_t)row * a.mat_stride, a.mat_begin, a.mat_end);
    TileCtx tc{hi_off, (1u << g.c) - 1, g.c};
    __syncthreads();
    const double2 *M = lm;  // offsets below are taken relative to mat_begin

    if (a.product_init) {
        // per-qubit product-state vectors: column 0 of each init matrix
        for (int j = threadIdx.x; j < (1 << a1) + (1 << (t - a1)); j += blockDim.x) {
            const bool first = j < (1 << a1);
            const int k0 = first ? 0 : a1, k1 = first ? a1 : t;
            const int v = first ? j : j - (1 << a1);
            double2 acc = make_double2(1.0, 0.0);
            for (int k = k0; k < k1; k++) {
                int pos = k < g.c ? k : g.hb[k - g.c];
                int q = g.n - 1 - pos;
                const double2 *im = M + (a.init_mat[q] - a.mat_begin);
                acc = zmul(acc, ((v >> (k - k0)) & 1) ? im[2] : im[0]);
            }
            if (first) p1[v] = acc;
            else p2[v] = acc;
        }
    }
    __syncthreads();

    const int64_t ntiles = (int64_t)1 << a.tiles_log2;
    for (int64_t tile = w; tile < ntiles; tile += a.wg_per_row) {
        const uint64_t fb = pdep64((uint64_t)tile, g.fixed_mask);
        if (a.product_init) {
            double2 f = make_double2(1.0, 0.0);
            for (uint64_t fm = g.fixed_mask; fm; fm &= fm - 1) {
                int pos = __ffsll((unsigned long long)fm) - 1;
                const double2 *im = M + (a.init_mat[g.n - 1 - pos] - a.mat_begin);
                f = zmul(f, ((fb >> pos) & 1) ? im[2] : im[0]);
            }
            for (int l = threadIdx.x; l < T; l += blockDim.x)
                lds[sw(l)] = down2(zmul(f, zmul(p1[l & ((1 << a1) - 1)], p2[l >> a1])));
        } else {
            tile_copy<true>(tc, lds, st, fb, T);
        }
        __syncthreads();
        for (int si = 0; si < a.nstages; si++) {
            const Stage st = cget(a.stages, si);
            run_stage_any(st, a.ops, M, a.mat_begin, smat(a.mats + (int64_t)row * a.mat_stride), lds, t, fb, threadIdx.x, blockDim.x);
            __syncthreads();
        }
        tile_copy<false>(tc, lds, st, fb, T);
        __syncthreads();
    }
}

// ------------------------------------------------- expectation partials
// Term t on a tile with fixed bits fb:
//   x == 0:   sum_l (-1)^{|g(l) & z|} |psi_l|^2
//   x != 0:   pairs (i, j = i ^ x) with bit m(x) of i clear contribute
//             2 Re(i^{ny} (-1)^{|j & z|} conj(psi_i) psi_j)
// where m is the lowest set bit of x's in-tile part (partner in LDS) or, when
// x flips fixed bits, of its out-of-tile part (partner tile in HBM, and only
// tiles with that bit clear count the pair).
__device__ __forceinline__ double re_iny(int ny, double s, double2 A)
{
    switch (ny & 3) {
    case 0: return s * A.x;
    case 1: return -s * A.y;
    case 2: return -s * A.x;
    default: return s * A.y;
    }
}

__device__ double term_tile_sum(const TermDev &tm, const TileCtx &tc, const float2 *lds, const float2 *row, uint64_t fb,
                                int t, int tid, int nt)
{
    const uint32_t T = 1u << t;
    double acc = 0;
    if (tm.x == 0) {
        const int zf = par64(fb & tm.z);
        for (uint32_t l = tid; l < T; l += nt) {
            double2 v = up2(lds[sw(l)]);
            double pr = v.x * v.x + v.y * v.y;
            acc += ((zf ^ par32(l & tm.zl)) ? -pr : pr);
        }
    } else if (tm.xout == 0) {
        const int zf = par64(fb & tm.z);
        const int mb = __ffs(tm.xl) - 1;
        for (uint32_t p = tid; p < T / 2; p += nt) {
            uint32_t i = ins0(p, mb), j = i ^ tm.xl;
            double2 a = up2(lds[sw(i)]), c = up2(lds[sw(j)]);
            double2 A = make_double2(a.x * c.x + a.y * c.y, a.x * c.y - a.y * c.x);  // conj(a) c
            double s = (zf ^ par32(j & tm.zl)) ? -2.0 : 2.0;
            acc += re_iny(tm.ny, s, A);
        }
    } else {
        const int mb = __ffsll((unsigned long long)tm.xout) - 1;
        if ((fb >> mb) & 1) return 0.0;
        const uint64_t fj = fb ^ tm.xout;
        const int zf = par64(fj & tm.z);
        for (uint32_t l = tid; l < T; l += nt) {
            uint32_t lj = l ^ tm.xl;
            double2 a = up2(lds[sw(l)]), c = up2(row[tile_index(tc, fj, lj)]);
            double2 A = make_double2(a.x * c.x + a.y * c.y, a.x * c.y - a.y * c.x);
            double s = (zf ^ par32(lj & tm.zl)) ? -2.0 : 2.0;
            acc += re_iny(tm.ny, s, A);
        }
    }
    return acc;
}

// --------------------------------------------------- phi = H_g psi
// (P psi)[i] = i^{ny} (-1)^{|(i ^ x) & z|} psi[i ^ x]; the coefficient of term
// t of observable k is upstream[b, k] * coeff_t.  One output element.
__device__ __forceinline__ float2 h_elem(uint32_t l, uint64_t fb, const TermDev *terms, int nterm, const float *up,
                                         const float2 *lds, const TileCtx &tc, const float2 *ps)
{
    double ax = 0, ay = 0;
    for (int k = 0; k < nterm; k++) {
        const TermDev tm = cget(terms, k);
        const uint32_t lj = l ^ tm.xl;
        const uint64_t fj = fb ^ tm.xout;
        float2 v = tm.xout == 0 ? lds[sw(lj)] : ps[tile_index(tc, fj, lj)];
        double cf = tm.coeff * (double)up[tm.k];
        if (par64(fj & tm.z) ^ par32(lj & tm.zl)) cf = -cf;
        double vx = v.x, vy = v.y;
        switch (tm.ny & 3) {
        case 0: ax += cf * vx; ay += cf * vy; break;
        case 1: ax -= cf * vy; ay += cf * vx; break;
        case 2: ax -= cf * vx; ay -= cf * vy; break;
        default: ax += cf * vy; ay -= cf * vx; break;
        }
    }
    return make_float2((float)ax, (float)ay);
}

// ------------------------------------------------ Pauli sums on tiles
// The hardware hands consecutive workgroup ids to the 8 XCDs in turn; this
// renumbering gives each XCD a contiguous range of (row, tile) work so that
// the tiles of one row, which read each other as partner tiles, share that
// XCD's L2.
__device__ __forceinline__ int xcd_block(int bid, int nb)
{
    if (nb % 8) return bid;
    return (bid % 8) * (nb / 8) + bid / 8;
}

// Expectations of Pauli sums, and optionally phi = sum_k g_k h_k psi, over
// tiles of T = 256 P amplitudes (T < 256 when P == 1: the state is smaller).
// Thread tid owns the amplitudes l = tid + 256 r of the tile.  For each x
// group the thread forms d(l) = sum_t c'_t chi_{z_t}(l) from the group's
// terms (one sign per term and thread, one per u sub-group and register),
// reads the partner amplitudes psi_{l ^ x} once, and adds
// Re(conj(psi_l) d(l) psi_{l ^ x}) to the group's observable and
// g_k d(l) psi_{l ^ x} to phi_l.  Accumulation is in fp64; each workgroup
// reduces its expectation partials in a fixed order.
template <int P, bool kPhi>
__global__ __launch_bounds__(256) void k_pauli(PauliArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const TileGeom &g = a.g;
    const int T = 1 << g.t;
    float2 *la = reinterpret_cast<float2 *>(smem);
    uint64_t *hi_off = reinterpret_cast<uint64_t *>(la + T);
    double *red = reinterpret_cast<double *>(hi_off + (1 << g.h));  // [kPauliChunk][4 waves]
    double *esum = red + 4 * kPauliChunk;                           // [k_count]
    float2 *lb = reinterpret_cast<float2 *>(esum + a.k_count);      // partner tile (when any xF != 0)

    const int bid = xcd_block(blockIdx.x, gridDim.x);
    const int row = bid / a.wg_per_row, w = bid % a.wg_per_row;
    const int b = cget(a.rows, row);
    const float2 *ps = a.psi + (int64_t)b * a.row_stride;
    const PChunk *chunks = a.chunks + cget(a.row_chunk_begin, row);
    const int nchunks = cget(a.row_chunk_count, row);
    const float *up = kPhi ? a.upstream + (int64_t)a.brows[row] * a.K : nullptr;
    const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64;
    const bool active = tid < T;
    const int kend = a.k_begin + a.k_count;
    build_hi_off(g, hi_off);
    for (int j = tid; j < a.k_count; j += blockDim.x) esum[j] = 0;
    TileCtx tc{hi_off, (1u << g.c) - 1, g.c};
    __syncthreads();

    const int64_t ntiles = (int64_t)1 << a.tiles_log2;
    for (int64_t tile = w; tile < ntiles; tile += a.wg_per_row) {
        const uint64_t fb = pdep64((uint64_t)tile, g.fixed_mask);
        tile_copy<true, (P > 1 ? P / 2 : 1)>(tc, la, const_cast<float2 *>(ps), fb, T);
        __syncthreads();
        float2 own[P];
#pragma unroll
        for (int r = 0; r < P; r++) own[r] = active ? la[sw(tid + 256 * r)] : make_float2(0.f, 0.f);
        double2 acc[kPhi ? P : 1];
#pragma unroll
        for (int r = 0; r < (kPhi ? P : 1); r++) acc[r] = make_double2(0.0, 0.0);

        for (int ci = 0; ci < nchunks; ci++) {
            const PChunk ch = cget(chunks, ci);
            if (ch.k0 < a.k_begin || ch.k0 >= kend) continue;
            double ek[kPauliChunk];
#pragma unroll
            for (int j = 0; j < kPauliChunk; j++) ek[j] = 0.0;
            for (int xi = ch.xf_begin; xi < ch.xf_end; xi++) {
                const PXfGroup xf = cget(a.xfg, xi);
                const float2 *src = la;
                if (xf.xF) {
                    __syncthreads();  // the previous partner tile is consumed
                    tile_copy<true, (P > 1 ? P / 2 : 1)>(tc, lb, const_cast<float2 *>(ps), fb ^ xf.xF, T);
                    __syncthreads();
                    src = lb;
                }
                for (int gi = xf.x_begin; gi < xf.x_end; gi++) {
                    const PXGroup xg = cget(a.xg, gi);
                    double dr[P], di[P];
#pragma unroll
                    for (int r = 0; r < P; r++) dr[r] = di[r] = 0.0;
                    for (int ui = xg.u_begin; ui < xg.u_end; ui++) {
                        const PUSub us = cget(a.us, ui);
                        double er = 0.0, ei = 0.0;
                        for (int ti = us.t_begin; ti < us.t_end; ti++) {
                            const PTerm tm = cget(a.terms, ti);
                            const double c = (par64(fb & tm.zF) ^ par32((uint32_t)tid & tm.zlo)) ? -tm.c : tm.c;
                            if (tm.im) ei += c;
                            else er += c;
                        }
#pragma unroll
                        for (int r = 0; r < P; r++) {
                            const double sg = (__popc(us.u & (uint32_t)r) & 1) ? -1.0 : 1.0;
                            dr[r] = fma(sg, er, dr[r]);
                            di[r] = fma(sg, ei, di[r]);
                        }
                    }
                    const bool self = xf.xF == 0 && xg.xT == 0;
                    const double gk = kPhi ? (double)up[ch.k0 + xg.kk] : 0.0;
                    double ex = 0.0;
                    if (!(xg.flags & 2)) {
#pragma unroll
                        for (int r = 0; r < P; r++) {
                            float2 pv = own[r];
                            if (!self && active) pv = src[sw((tid + 256 * r) ^ xg.xT)];
                            const double tr = dr[r] * (double)pv.x, ti = dr[r] * (double)pv.y;
                            ex = fma((double)own[r].x, tr, fma((double)own[r].y, ti, ex));
                            if (kPhi) {
                                acc[r].x = fma(gk, tr, acc[r].x);
                                acc[r].y = fma(gk, ti, acc[r].y);
                            }
                        }
                    } else {
#pragma unroll
                        for (int r = 0; r < P; r++) {
                            float2 pv = own[r];
                            if (!self && active) pv = src[sw((tid + 256 * r) ^ xg.xT)];
                            const double px = pv.x, py = pv.y;
                            const double tr = fma(dr[r], px, -di[r] * py), ti = fma(dr[r], py, di[r] * px);
                            ex = fma((double)own[r].x, tr, fma((double)own[r].y, ti, ex));
                            if (kPhi) {
                                acc[r].x = fma(gk, tr, acc[r].x);
                                acc[r].y = fma(gk, ti, acc[r].y);
                            }
                        }
                    }
#pragma unroll
                    for (int j = 0; j < kPauliChunk; j++) ek[j] += (j == xg.kk) ? ex : 0.0;
                }
            }
            // this tile's share of the chunk's expectations, in a fixed order
#pragma unroll
            for (int j = 0; j < kPauliChunk; j++)
                if (j < ch.nk) {
                    const double v = wave_sum(ek[j]);
                    if (lane == 0) red[j * 4 + wave] = v;
                }
            __syncthreads();
            if (tid < ch.nk)
                esum[ch.k0 - a.k_begin + tid] += ((red[tid * 4] + red[tid * 4 + 1]) + red[tid * 4 + 2]) + red[tid * 4 + 3];
            __syncthreads();
        }
        if (kPhi && active) {
            float2 *ph = a.phi + (int64_t)b * a.row_stride;
#pragma unroll
            for (int r = 0; r < P; r++) {
                const uint64_t i = tile_index(tc, fb, tid + 256 * r);
                double2 v = acc[r];
                if (a.phi_accumulate) v = zadd(v, up2(ph[i]));
                ph[i] = down2(v);
            }
        }
        __syncthreads();
    }
    double *out = a.partial + ((int64_t)row * a.wg_per_row + w) * a.k_count;
    for (int j = tid; j < a.k_count; j += blockDim.x) out[j] = esum[j];
}

// out[b, k] = sum over the row's workgroups of their partials: one block per
// (row, observable), strided sums then a tree, all in a fixed order.
__global__ __launch_bounds__(256) void k_pauli_reduce(PauliReduceArgs a)
{
    __shared__ double red[256];
    const int row = blockIdx.x, j = blockIdx.y;
    const double *p = a.partial + (int64_t)row * a.wg_per_row * a.k_count + j;
    double s = 0;
    for (int w = threadIdx.x; w < a.wg_per_row; w += blockDim.x) s += p[(int64_t)w * a.k_count];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
        __syncthreads();
    }
    if (threadIdx.x == 0) a.out[(int64_t)a.rows[row] * a.K + a.k_begin + j] = (float)red[0];
}

// ------------------------------------------ diagonal Pauli sums in HBM
// Expectations of Z-only Pauli sums, streamed from HBM without LDS staging:
// workgroup w of a row sweeps the blocks w, w + wg_per_row, ... of the row,
// loading each thread's 16 amplitudes of the next block while it transforms
// the current one.  The class weights D(blk) are staged in LDS for
// kDiagRefill blocks at a time (a wave per class, a lane per block; classes
// past the chunk's get weight zero, so every block runs the same straight-line
// code).  Class c
// accumulates D(blk) W_v in its own register; the thread's sign chi_zT(tid)
// is applied once at the end, before the fixed-order reduction of each
// observable.
template <int A>
__global__ __launch_bounds__(256) void k_pauli_diag(DiagArgs a)
{
    __shared__ double dw[A * kDiagRefill];
    __shared__ double red[4];
    extern __shared__ __align__(16) unsigned char smem[];
    double *esum = reinterpret_cast<double *>(smem);  // [k_count]

    const int bid = xcd_block(blockIdx.x, gridDim.x);
    const int row = bid / a.wg_per_row, w = bid % a.wg_per_row;
    const int b = cget(a.rows, row);
    const float4 *ps = reinterpret_cast<const float4 *>(a.psi + (int64_t)b * a.row_stride);
    const int tid = threadIdx.x, lane = tid % 64;
    const int wave = __builtin_amdgcn_readfirstlane(tid / 64);
    // blocks of this workgroup: w + i wg_per_row for i < mine (w < wg_per_row <= blocks)
    const int64_t mine = (((int64_t)1 << a.blocks_log2) - w + a.wg_per_row - 1) / a.wg_per_row;
    const int kend = a.k_begin + a.k_count;
    const DChunk *chunks = a.chunks + cget(a.row_chunk_begin, row);
    const int nchunks = cget(a.row_chunk_count, row);
    for (int j = tid; j < a.k_count; j += blockDim.x) esum[j] = 0;

    for (int ci = 0; ci < nchunks; ci++) {
        const DChunk ch = cget(chunks, ci);
        if (ch.k_hi < a.k_begin || ch.k_lo >= kend) continue;
        const DClass *cls = a.classes + ch.c_begin;
        const int ncls = ch.c_end - ch.c_begin;
        double G[A];
        uint32_t vv[A];
#pragma unroll
        for (int c = 0; c < A; c++) {
            G[c] = 0.0;
            vv[c] = c < ncls ? cget(cls, c).v : 0u;
        }
        float4 nx[8];
        auto load = [&](int64_t i) {
            const float4 *src = ps + ((w + i * a.wg_per_row) << (kDiagBlockBits - 1)) + tid;
#pragma unroll
            for (int j = 0; j < 8; j++) nx[j] = src[256 * j];
        };
        load(0);
        for (int64_t i = 0; i < mine; i++) {
            const int slot = (int)(i % kDiagRefill);
            if (slot == 0) {
                __syncthreads();  // the previous weights are consumed
                const uint64_t blk = (uint64_t)(w + (i + lane) * a.wg_per_row);
                for (int c = wave; c < A; c += 4) {
                    double d = 0.0;  // classes past the chunk's weigh nothing
                    if (c < ncls) {
                        const DClass cc = cget(cls, c);
                        for (int t = cc.t_begin; t < cc.t_end; t++) {
                            const DTerm tm = cget(a.terms, t);
                            d += par64(blk & tm.zB) ? -tm.c : tm.c;
                        }
                    }
                    dw[lane * A + c] = d;
                }
                __syncthreads();
            }
            double p[16];
#pragma unroll
            for (int j = 0; j < 8; j++) {
                p[2 * j] = fma((double)nx[j].x, (double)nx[j].x, (double)nx[j].y * (double)nx[j].y);
                p[2 * j + 1] = fma((double)nx[j].z, (double)nx[j].z, (double)nx[j].w * (double)nx[j].w);
            }
            if (i + 1 < mine) load(i + 1);
            // Walsh transform over the four register bits: p[v] = W_v
#pragma unroll
            for (int sb = 1; sb < 16; sb <<= 1)
#pragma unroll
                for (int r = 0; r < 16; r++)
                    if (!(r & sb)) {
                        const double x = p[r], y = p[r | sb];
                        p[r] = x + y;
                        p[r | sb] = x - y;
                    }
            double dv[A];
#pragma unroll
            for (int c = 0; c < A; c++) dv[c] = dw[slot * A + c];
#pragma unroll
            for (int c = 0; c < A; c++) G[c] = fma(dv[c], p[vv[c]], G[c]);
        }
        // thread signs, then one fixed-order reduction per observable
        const int k_first = ch.k_lo > a.k_begin ? ch.k_lo : a.k_begin;
        const int k_last = ch.k_hi < kend - 1 ? ch.k_hi : kend - 1;
        for (int k = k_first; k <= k_last; k++) {
            double e = 0.0;
#pragma unroll
            for (int c = 0; c < A; c++)
                if (c < ncls) {
                    const DClass cc = cget(cls, c);
                    if (cc.k == k) e += par32((uint32_t)tid & cc.zT) ? -G[c] : G[c];
                }
            const double v = wave_sum(e);
            if (lane == 0) red[wave] = v;
            __syncthreads();
            if (tid == 0) esum[k - a.k_begin] += ((red[0] + red[1]) + red[2]) + red[3];
            __syncthreads();
        }
    }
    __syncthreads();
    double *out = a.partial + ((int64_t)row * a.wg_per_row + w) * a.k_count;
    for (int j = tid; j < a.k_count; j += blockDim.x) out[j] = esum[j];
}

// ------------------------------------------------------ reverse pass
// psi and phi tiles side by side in LDS; the pass's matrices too.
__global__ __launch_bounds__(256, 2) void k_rev_pass(RevArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const TileGeom &g = a.g;
    const int t = g.t;
    const uint32_t T = 1u << t;
    float2 *lp = reinterpret_cast<float2 *>(smem);
    float2 *lf = lp + T;
    uint64_t *hi_off = reinterpret_cast<uint64_t *>(lf + T);
    double2 *lm = reinterpret_cast<double2 *>(hi_off + (1 << g.h));
    double *acc = reinterpret_cast<double *>(lm + (a.mat_end - a.mat_begin));  // [4][gcount]

    const int row = blockIdx.x / a.wg_per_row, w = blockIdx.x % a.wg_per_row;
    const int b = cget(a.rows, row);
    float2 *sp = a.psi + (int64_t)b * a.row_stride;
    float2 *sf = a.phi + (int64_t)b * a.row_stride;
    build_hi_off(g, hi_off);
    stage_mats(lm, a.mats + (int64_t)row * a.mat_stride, a.mat_begin, a.mat_end);
    for (int j = threadIdx.x; j < 4 * a.gcount; j += blockDim.x) acc[j] = 0;
    TileCtx tc{hi_off, (1u << g.c) - 1, g.c};
    const int tid = threadIdx.x, nt = blockDim.x;
    __syncthreads();

    const int64_t ntiles = (int64_t)1 << a.tiles_log2;
    for (int64_t tile = w; tile < ntiles; tile += a.wg_per_row) {
        const uint64_t fb = pdep64((uint64_t)tile, g.fixed_mask);
        tile_copy<true>(tc, lp, sp, fb, T);
        tile_copy<true>(tc, lf, sf, fb, T);
        __syncthreads();
        for (int si = 0; si < a.nstages; si++) {
            const Stage st = cget(a.stages, si);
            run_rev_stage_any<kStageBitsRev>(st, a.ops, lm, a.mat_begin, lp, lf, t, fb, acc, a.gcount, a.gbase, threadIdx.x, blockDim.x);
            __syncthreads();
        }
        if (a.store) {
            tile_copy<false>(tc, lp, sp, fb, T);
            tile_copy<false>(tc, lf, sf, fb, T);
        }
        __syncthreads();
    }
    double *out = a.gpart + ((int64_t)row * a.wg_per_row + w) * a.n_gslots + a.gbase;
    for (int j = tid; j < a.gcount; j += nt)
        out[j] = ((acc[j] + acc[a.gcount + j]) + acc[2 * a.gcount + j]) + acc[3 * a.gcount + j];
}

// grad[b, s] = sum over gradient slots of s: 2 * scale * sum_w gpart
__global__ void k_grad_reduce(GradReduceArgs a)
{
    const int row = blockIdx.x;
    const int b = cget(a.rows, row);
    const double *scale = a.slot_scale + (a.uniform ? 0 : (int64_t)row * a.n_slots);
    const double *p = a.gpart + (int64_t)row * a.wg_per_row * a.n_gslots;
    for (int s = threadIdx.x; s < a.S; s += blockDim.x) {
        double sum = 0;
        for (int k = a.sym_begin[s]; k < a.sym_begin[s + 1]; k++) {
            int gs = a.sym_gslots[k];
            double v = 0;
            for (int w = 0; w < a.wg_per_row; w++) v += p[(int64_t)w * a.n_gslots + gs];
            sum += 2.0 * scale[a.gslot_slot[gs]] * v;
        }
        a.grad[(int64_t)b * a.S + s] = (float)sum;
    }
}

// ---------------------------------------------------- resident circuits
// Small circuits (psi, phi and every matrix of the row fit in LDS): one
// workgroup per batch row does the whole call -- product-state init, forward
// gates, expectations, H_g, reverse sweep, gradient reduction -- in one
// launch, on the matrices k_build_mats wrote.  At most 128 registers per
// thread, so that four rows share a CU.  Outputs are reduced in a fixed order.
// The resident computation in three parts around the forward and reverse
// register stages (which the generic kernel loops over and a specialised
// kernel spells out).  acc: one accumulator row per wave (terms, then
// gradient slots); lp/lf: psi/phi of the row in LDS.
template <class MT>
__device__ __forceinline__ void resident_begin(const ResArgs &a, MT M, double *acc, float2 *lp, int tid, int nt)
{
    const int n = a.n;
    const uint32_t T = 1u << n;
    for (int j = tid; j < (nt / 64) * a.nacc; j += nt) acc[j] = 0;
    // product-state initialisation
    for (uint32_t l = tid; l < T; l += nt) {
        double2 v = make_double2(1.0, 0.0);
        for (int q = 0; q < n; q++) v = zmul(v, M[a.init_mat[q] + (((l >> (n - 1 - q)) & 1) ? 2 : 0)]);
        lp[sw(l)] = down2(v);
    }
    __syncthreads();
}

// state output, expectation terms, and (adjoint) phi = H_g psi
__device__ __forceinline__ void resident_middle(const ResArgs &a, double *acc, float2 *lp, float2 *lf, int row, int tid, int nt)
{
    const int n = a.n;
    const uint32_t T = 1u << n;
    const int b = cget(a.rows, row);
    const int wave = tid / 64, lane = tid % 64;
    // whole-state tile: every term's partner is local, so the tile index
    // table and the HBM partner pointer are never used (valid LDS addresses
    // are passed instead of null pointers)
    TileCtx tc{reinterpret_cast<const uint64_t *>(acc), T - 1, n};
    if (a.state_out) {
        float2 *out = a.state_out + (int64_t)a.out_rows[row] * a.out_stride;
        for (uint32_t l = tid; l < T; l += nt) out[l] = lp[sw(l)];
    }
    const TermDev *terms = a.terms ? a.terms + cget(a.row_term_begin, row) : nullptr;
    const int nterm = a.terms ? cget(a.row_term_count, row) : 0;
    for (int k = 0; k < nterm; k++) {
        double v = wave_sum(term_tile_sum(cget(terms, k), tc, lp, lp, 0, n, tid, nt));
        if (lane == 0) acc[wave * a.nacc + k] += v;
    }
    if (a.grad) {
        const float *up = a.upstream + (int64_t)b * a.K;
        for (uint32_t l = tid; l < T; l += nt) lf[sw(l)] = h_elem(l, 0, terms, nterm, up, lp, tc, lp);
        __syncthreads();
    }
}

// outputs: expectations and gradients, reduced over the waves in a fixed order
__device__ __forceinline__ void resident_end(const ResArgs &a, double *acc, int row, int tid, int nt)
{
    __syncthreads();
    const int b = cget(a.rows, row);
    const int nw = nt / 64;
    const TermDev *terms = a.terms ? a.terms + cget(a.row_term_begin, row) : nullptr;
    const int nterm = a.terms ? cget(a.row_term_count, row) : 0;
    auto total = [&](int j) {
        double s = 0;
        for (int w = 0; w < nw; w++) s += acc[w * a.nacc + j];
        return s;
    };
    if (a.exp_out)
        for (int k = tid; k < a.K; k += nt) {
            double sum = 0;
            for (int ti = 0; ti < nterm; ti++) {
                const TermDev tm = cget(terms, ti);
                if (tm.k == k) sum += tm.coeff * total(ti);
            }
            a.exp_out[(int64_t)b * a.K + k] = (float)sum;
        }
    if (a.grad) {
        const double *scale = a.slot_scale + (a.uniform ? 0 : (int64_t)row * a.n_slots);
        for (int s = tid; s < a.S; s += nt) {
            double sum = 0;
            for (int k = a.sym_begin[s]; k < a.sym_begin[s + 1]; k++) {
                const int gs = a.sym_gslots[k];
                sum += 2.0 * scale[a.gslot_slot[gs]] * total(a.gacc + gs);
            }
            a.grad[(int64_t)b * a.S + s] = (float)sum;
        }
    }
}

__global__ __launch_bounds__(256, 4) void k_resident(ResArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const uint32_t T = 1u << a.n;
    double *acc = reinterpret_cast<double *>(smem);              // [4][nacc]
    float2 *lp = reinterpret_cast<float2 *>(acc + 4 * a.nacc);   // [T]
    float2 *lf = lp + T;                                         // [T] (adjoint)
    const SMat M = smat(a.mats + (int64_t)blockIdx.x * a.mat_stride);
    const int tid = threadIdx.x, nt = blockDim.x;
    resident_begin(a, M, acc, lp, tid, nt);
    for (int si = 0; si < a.nfstages; si++) {
        const Stage st = cget(a.fstages, si);
        run_stage_any(st, a.fops, M, 0, M, lp, a.n, 0, tid, nt);
        __syncthreads();
    }
    resident_middle(a, acc, lp, lf, blockIdx.x, tid, nt);
    if (a.grad)
        for (int si = 0; si < a.nrstages; si++) {
            const Stage st = cget(a.rstages, si);
            run_rev_stage_any<kStageBitsRevResident>(st, a.rops, M, 0, lp, lf, a.n, 0, acc, a.nacc, -a.gacc, tid, nt);
            __syncthreads();
        }
    resident_end(a, acc, blockIdx.x, tid, nt);
}

// ------------------------------------------------------------- sampling
__device__ __forceinline__ uint64_t weight_of(float2 v)
{
    double re = v.x, im = v.y;
    double p = re * re + im * im;
    return (uint64_t)(p * 0x1p62);
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v)
{
    for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
    return v;
}

// level 1: sum of the weights of each group of 64 amplitudes
__global__ __launch_bounds__(256) void k_samp_l1(SampArgs a)
{
    const int row = blockIdx.y;
    const int sr = a.rows ? a.rows[row] : row;
    const int64_t grp = (int64_t)blockIdx.x * 4 + threadIdx.x / 64;
    const int lane = threadIdx.x % 64;
    if (grp >= a.count[1]) return;
    const int64_t i = grp * 64 + lane;
    const float2 *st = a.state + (int64_t)sr * a.row_stride;
    uint64_t wv = i < a.count[0] ? weight_of(st[i]) : 0;
    wv = wave_sum_u64(wv);
    if (lane == 0) a.levels[(int64_t)row * a.row_level + a.off[1] + grp] = wv;
}

// level k+1 from level k
__global__ __launch_bounds__(256) void k_samp_up(SampArgs a, int k)
{
    const int row = blockIdx.y;
    const int64_t grp = (int64_t)blockIdx.x * 4 + threadIdx.x / 64;
    const int lane = threadIdx.x % 64;
    if (grp >= a.count[k + 1]) return;
    const int64_t i = grp * 64 + lane;
    const uint64_t *lv = a.levels + (int64_t)row * a.row_level;
    uint64_t wv = i < a.count[k] ? lv[a.off[k] + i] : 0;
    wv = wave_sum_u64(wv);
    if (lane == 0) a.levels[(int64_t)row * a.row_level + a.off[k + 1] + grp] = wv;
}

// SplitMix64 (Steele, Lea, Flood 2014): output number `counter` of the stream
// whose state starts at `seed`
__device__ __forceinline__ uint64_t splitmix64(uint64_t seed, uint64_t counter)
{
    uint64_t z = seed + (counter + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// one wavefront per shot: descend the levels, at each one locating the child
// whose cumulative interval contains r by a wavefront prefix scan
__global__ __launch_bounds__(256) void k_samp_shots(SampArgs a)
{
    const int row = blockIdx.y;
    const int sr = a.rows ? a.rows[row] : row;
    const int b = a.brows ? a.brows[row] : row;
    const int64_t shot = (int64_t)blockIdx.x * 4 + threadIdx.x / 64;
    const int lane = threadIdx.x % 64;
    if (shot >= a.n_shots) return;
    const uint64_t *lv = a.levels + (int64_t)row * a.row_level;
    const float2 *st = a.state + (int64_t)sr * a.row_stride;
    const int top = a.nlev;
    auto level_value = [&](int k, int64_t i) -> uint64_t {
        if (i >= a.count[k]) return 0;
        return k == 0 ? weight_of(st[i]) : lv[a.off[k] + i];
    };
    // total weight from the top level (at most 64 entries)
    const uint64_t tv = level_value(top, lane);
    const uint64_t W = wave_sum_u64(tv);
    uint64_t *out = a.out + (int64_t)b * a.n_shots + shot;
    if (W == 0) {
        if (lane == 0) *out = 0;
        return;
    }
    const uint64_t u = splitmix64(a.seed, (uint64_t)b * (uint64_t)a.n_shots + (uint64_t)shot);
    uint64_t r = __umul64hi(u, W);
    int64_t base = 0;  // index of the chosen entry at the current level
    for (int k = top; k >= 0; k--) {
        const uint64_t v = k == top ? tv : level_value(k, base * 64 + lane);
        uint64_t incl = v;
        for (int d = 1; d < 64; d <<= 1) {
            uint64_t o = __shfl_up(incl, d, 64);
            if (lane >= d) incl += o;
        }
        const uint64_t hit = __ballot(incl > r);
        // the children of the chosen entry sum to its value (> r), so some lane
        // hits; the clamp only keeps indexing in range
        const int sel = hit ? __ffsll((unsigned long long)hit) - 1 : 63;
        const uint64_t before = __shfl(incl - v, sel, 64);
        r -= before;
        base = base * 64 + sel;
    }
    if (lane == 0) *out = (uint64_t)base;
}

// ------------------------------------------------------- gather, padding
__global__ void k_gather(GatherArgs a)
{
    const int row = blockIdx.y;
    const int b = a.brows ? a.brows[row] : row;
    const int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (m >= a.M) return;
    const uint64_t x = a.bits[(int64_t)b * a.M + m];
    float2 v = make_float2(0.f, 0.f);
    if ((x >> a.n) == 0) v = a.state[(int64_t)(a.rows ? a.rows[row] : row) * a.row_stride + (int64_t)x];
    a.out[(int64_t)b * a.M + m] = v;
}

__global__ void k_zero_tail(float2 *state, int64_t row_stride, const int32_t *rows, int64_t from, int64_t to)
{
    const int row = blockIdx.y;
    const int64_t i = from + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < to) state[(int64_t)rows[row] * row_stride + i] = make_float2(0.f, 0.f);
}

// ------------------------------------------------------- launch wrappers
// Opt-in profiler: launches of the selected kernel are bracketed by a pair
// of HIP events recorded on the launch stream.
namespace prof {
std::mutex mu;
std::string target;
std::vector<std::pair<hipEvent_t, hipEvent_t>> events;

struct Scope {
    hipEvent_t b = nullptr, e = nullptr;
    hipStream_t s;
    Scope(const char *name, hipStream_t st) : s(st)
    {
        std::lock_guard<std::mutex> l(mu);
        if (target.empty() || target != name) return;
        if (hipEventCreate(&b) != hipSuccess || hipEventCreate(&e) != hipSuccess) {
            b = e = nullptr;
            return;
        }
        (void)hipEventRecord(b, s);
    }
    ~Scope()
    {
        if (!b) return;
        (void)hipEventRecord(e, s);
        std::lock_guard<std::mutex> l(mu);
        events.emplace_back(b, e);
    }
};
} // namespace prof

void profile_start(const char *kernel)
{
    std::lock_guard<std::mutex> l(prof::mu);
    prof::target = kernel ? kernel : "";
}

hipError_t profile_read(int64_t *launches, double *total_ms)
{
    std::lock_guard<std::mutex> l(prof::mu);
    double tot = 0;
    hipError_t err = hipSuccess;
    for (auto &pe : prof::events) {
        float ms = 0;
        hipError_t e = hipEventSynchronize(pe.second);
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, pe.first, pe.second);
        if (e != hipSuccess) err = e;
        tot += ms;
    }
    *launches = (int64_t)prof::events.size();
    *total_ms = tot;
    for (auto &pe : prof::events) {
        (void)hipEventDestroy(pe.first);
        (void)hipEventDestroy(pe.second);
    }
    prof::events.clear();
    return err;
}

namespace {
template <class K> hipError_t set_lds(K kernel, size_t bytes)
{
    if (bytes <= 65536) return hipSuccess;
    return hipFuncSetAttribute(reinterpret_cast<const void *>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)bytes);
}
} // namespace

hipError_t launch_build_stage(const StageBuildArgs &a, int nrows, hipStream_t s)
{
    if (a.nlist <= 0 || nrows <= 0) return hipSuccess;
    prof::Scope ps("build", s);
    hipLaunchKernelGGL(k_build_stage, dim3(a.nlist, nrows), dim3(64), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_build(const BuildArgs &a, int nrows, hipStream_t s)
{
    int n = a.task_end - a.task_begin;
    if (n <= 0 || nrows <= 0) return hipSuccess;
    dim3 grid((n + 255) / 256, nrows);
    prof::Scope ps("build", s);
    hipLaunchKernelGGL(k_build_mats, grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

size_t pass_lds_bytes(const TileGeom &g, bool product_init, int nmat)
{
    size_t b = sizeof(float2) * ((size_t)1 << g.t) + sizeof(uint64_t) * ((size_t)1 << g.h) + sizeof(double2) * nmat;
    if (product_init) b += sizeof(double2) * (((size_t)1 << (g.t / 2)) + ((size_t)1 << (g.t - g.t / 2)));
    return b;
}

hipError_t launch_pass(const PassArgs &a, int nrows, hipStream_t s)
{
    size_t lds = pass_lds_bytes(a.g, a.product_init != 0, a.mat_end - a.mat_begin);
    hipError_t e = set_lds(k_pass, lds);
    if (e != hipSuccess) return e;
    prof::Scope ps("pass", s);
    hipLaunchKernelGGL(k_pass, dim3(nrows * a.wg_per_row), dim3(kThreads), lds, s, a);
    return hipGetLastError();
}

size_t pauli_lds_bytes(const TileGeom &g, int k_count, bool partner)
{
    return sizeof(float2) * ((size_t)1 << g.t) * (partner ? 2 : 1) + sizeof(uint64_t) * ((size_t)1 << g.h) +
           sizeof(double) * (4 * kPauliChunk + (size_t)k_count);
}

template <int P>
hipError_t launch_pauli_p(const PauliArgs &a, int nrows, size_t lds, hipStream_t s)
{
    const dim3 grid(nrows * a.wg_per_row);
    if (a.phi) {
        hipError_t e = set_lds(k_pauli<P, true>, lds);
        if (e != hipSuccess) return e;
        prof::Scope ps("pauli", s);
        hipLaunchKernelGGL((k_pauli<P, true>), grid, dim3(kThreads), lds, s, a);
    } else {
        hipError_t e = set_lds(k_pauli<P, false>, lds);
        if (e != hipSuccess) return e;
        prof::Scope ps("pauli", s);
        hipLaunchKernelGGL((k_pauli<P, false>), grid, dim3(kThreads), lds, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_pauli(const PauliArgs &a, int nrows, bool partner, hipStream_t s)
{
    if (nrows <= 0) return hipSuccess;
    const size_t lds = pauli_lds_bytes(a.g, a.k_count, partner);
    switch (a.g.t <= 8 ? 1 : 1 << (a.g.t - 8)) {
    case 1: return launch_pauli_p<1>(a, nrows, lds, s);
    case 2: return launch_pauli_p<2>(a, nrows, lds, s);
    case 4: return launch_pauli_p<4>(a, nrows, lds, s);
    case 8: return launch_pauli_p<8>(a, nrows, lds, s);
    case 16: return launch_pauli_p<16>(a, nrows, lds, s);
    default: return hipErrorInvalidValue;
    }
}

template <int A> hipError_t launch_pauli_diag_a(const DiagArgs &a, int nrows, hipStream_t s)
{
    const size_t lds = sizeof(double) * (size_t)a.k_count;
    hipError_t e = set_lds(k_pauli_diag<A>, lds);
    if (e != hipSuccess) return e;
    prof::Scope ps("pauli", s);
    hipLaunchKernelGGL(k_pauli_diag<A>, dim3(nrows * a.wg_per_row), dim3(kThreads), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_pauli_diag(const DiagArgs &a, int nrows, int amax, hipStream_t s)
{
    if (nrows <= 0) return hipSuccess;
    if (amax <= 8) return launch_pauli_diag_a<8>(a, nrows, s);
    if (amax <= 16) return launch_pauli_diag_a<16>(a, nrows, s);
    return launch_pauli_diag_a<kDiagClassMax>(a, nrows, s);
}

hipError_t launch_pauli_reduce(const PauliReduceArgs &a, int nrows, hipStream_t s)
{
    if (nrows <= 0 || a.k_count <= 0) return hipSuccess;
    prof::Scope ps("pauli_reduce", s);
    hipLaunchKernelGGL(k_pauli_reduce, dim3(nrows, a.k_count), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_rev_pass(const RevArgs &a, int nrows, hipStream_t s)
{
    size_t lds = 2 * sizeof(float2) * ((size_t)1 << a.g.t) + sizeof(uint64_t) * ((size_t)1 << a.g.h) +
                 sizeof(double2) * (size_t)(a.mat_end - a.mat_begin) + sizeof(double) * 4 * (size_t)(a.gcount > 0 ? a.gcount : 1);
    hipError_t e = set_lds(k_rev_pass, lds);
    if (e != hipSuccess) return e;
    prof::Scope ps("rev_pass", s);
    hipLaunchKernelGGL(k_rev_pass, dim3(nrows * a.wg_per_row), dim3(kThreads), lds, s, a);
    return hipGetLastError();
}

size_t resident_lds_bytes(int n, int nacc, bool adjoint)
{
    return sizeof(double) * 4 * (size_t)nacc + sizeof(float2) * ((size_t)1 << n) * (adjoint ? 2 : 1);
}

hipError_t launch_resident(const ResArgs &a, int nrows, hipStream_t s)
{
    if (nrows <= 0) return hipSuccess;
    size_t lds = resident_lds_bytes(a.n, a.nacc, a.grad != nullptr);
    hipError_t e = set_lds(k_resident, lds);
    if (e != hipSuccess) return e;
    prof::Scope ps("resident", s);
    hipLaunchKernelGGL(k_resident, dim3(nrows), dim3(kThreads), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_grad_reduce(const GradReduceArgs &a, int nrows, hipStream_t s)
{
    prof::Scope ps("grad_reduce", s);
    hipLaunchKernelGGL(k_grad_reduce, dim3(nrows), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_sample(const SampArgs &a, int nrows, hipStream_t s)
{
    if (nrows <= 0) return hipSuccess;
    if (a.nlev >= 1) {
        {
            prof::Scope ps("samp_l1", s);
            hipLaunchKernelGGL(k_samp_l1, dim3((unsigned)((a.count[1] + 3) / 4), nrows), dim3(256), 0, s, a);
        }
        for (int k = 1; k < a.nlev; k++)
            hipLaunchKernelGGL(k_samp_up, dim3((unsigned)((a.count[k + 1] + 3) / 4), nrows), dim3(256), 0, s, a, k);
    }
    if (a.n_shots > 0) {
        prof::Scope ps("samp_shots", s);
        hipLaunchKernelGGL(k_samp_shots, dim3((unsigned)((a.n_shots + 3) / 4), nrows), dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_gather(const GatherArgs &a, int nrows, hipStream_t s)
{
    if (a.M <= 0 || nrows <= 0) return hipSuccess;
    prof::Scope ps("gather", s);
    hipLaunchKernelGGL(k_gather, dim3((unsigned)((a.M + 255) / 256), nrows), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_zero_tail(float2 *state, int64_t row_stride, const int32_t *rows, int nrows, int64_t from, int64_t to,
                            hipStream_t s)
{
    if (to <= from || nrows <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_zero_tail, dim3((unsigned)((to - from + 255) / 256), nrows), dim3(256), 0, s, state,
                       row_stride, rows, from, to);
    return hipGetLastError();
}

} // namespace tq
