// device_ops.h -- device code shared by the precompiled kernels of libtq
// and by the kernels it specialises for one circuit structure at run time:
// arithmetic helpers, tile access, register-level gate ops and stages, Pauli
// term sums, and the parts of the resident-circuit computation.  It includes
// no host headers, so that the run-time compiler can take it as it is.
#pragma once
#include "kernel_args.h"

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
// m0 a0 + m1 a1 + m2 a2 + m3 a3: one multiply and seven FMAs per component
__device__ __forceinline__ double2 zmul4(double2 m0, double2 a0, double2 m1, double2 a1, double2 m2, double2 a2,
                                         double2 m3, double2 a3)
{
    return make_double2(m0.x * a0.x - m0.y * a0.y + m1.x * a1.x - m1.y * a1.y + m2.x * a2.x - m2.y * a2.y +
                            m3.x * a3.x - m3.y * a3.y,
                        m0.x * a0.y + m0.y * a0.x + m1.x * a1.y + m1.y * a1.x + m2.x * a2.y + m2.y * a2.x +
                            m3.x * a3.y + m3.y * a3.x);
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
    o.v00 = zmul2(a, v.v00, bs, v.v11);
    o.v11 = zmul2(a, v.v11, bs, v.v00);
    o.v01 = zmul2(a, v.v01, b, v.v10);
    o.v10 = zmul2(a, v.v10, b, v.v01);
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

// The same diagonal ops when some entries are known to be exactly 1 (bit k
// of U: entry k; its amplitudes are left as they are) or, for derivatives,
// exactly 0 (bit k of Z: entry k contributes nothing).
template <int R, int J, int U> __device__ __forceinline__ void rd1u(double2 *a, double2 e0, double2 e1)
{
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        const int idx = (k >> J) & 1;
        if ((U >> idx) & 1) continue;
        a[k] = zmul(idx ? e1 : e0, a[k]);
    }
}
template <int R, int J, int Z> __device__ __forceinline__ double rd1_dotz(const double2 *a, const double2 *f, double2 e0, double2 e1)
{
    double s = 0;
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        const int idx = (k >> J) & 1;
        if ((Z >> idx) & 1) continue;
        s += zdotr(f[k], zmul(idx ? e1 : e0, a[k]));
    }
    return s;
}
template <int R, int LO, int HI, int U>
__device__ __forceinline__ void rd2u(double2 *a, double2 e0, double2 e1, double2 e2, double2 e3)
{
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        const int idx = 2 * ((k >> LO) & 1) + ((k >> HI) & 1);
        if ((U >> idx) & 1) continue;
        a[k] = zmul(idx == 0 ? e0 : idx == 1 ? e1 : idx == 2 ? e2 : e3, a[k]);
    }
}
template <int R, int LO, int HI, int Z>
__device__ __forceinline__ double rd2_dotz(const double2 *a, const double2 *f, double2 e0, double2 e1, double2 e2, double2 e3)
{
    double s = 0;
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        const int idx = 2 * ((k >> LO) & 1) + ((k >> HI) & 1);
        if ((Z >> idx) & 1) continue;
        s += zdotr(f[k], zmul(idx == 0 ? e0 : idx == 1 ? e1 : idx == 2 ? e2 : e3, a[k]));
    }
    return s;
}

// dense 2x2 with a real matrix (imaginary parts exactly 0: RY, H and their
// products) on register bit J: half the arithmetic of rm1
template <int R, int J, class MT> __device__ __forceinline__ void rm1r(double2 *a, MT m)
{
    const double m00 = m[0].x, m01 = m[1].x, m10 = m[2].x, m11 = m[3].x;
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if ((k >> J) & 1) continue;
        const int kk = k | (1 << J);
        const double2 x = a[k], y = a[kk];
        a[k] = make_double2(fma(m00, x.x, m01 * y.x), fma(m00, x.y, m01 * y.y));
        a[kk] = make_double2(fma(m10, x.x, m11 * y.x), fma(m10, x.y, m11 * y.y));
    }
}
// dense 2x2 with real diagonal and imaginary off-diagonal entries (RX and its
// products; their real parts, resp. imaginary parts, are exactly 0) on
// register bit J: half the arithmetic of rm1
template <int R, int J, class MT> __device__ __forceinline__ void rm1x(double2 *a, MT m)
{
    const double d0 = m[0].x, o01 = m[1].y, o10 = m[2].y, d1 = m[3].x;
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if ((k >> J) & 1) continue;
        const int kk = k | (1 << J);
        const double2 x = a[k], y = a[kk];
        a[k] = make_double2(fma(d0, x.x, -o01 * y.y), fma(d0, x.y, o01 * y.x));
        a[kk] = make_double2(fma(d1, y.x, -o10 * x.y), fma(d1, y.y, o10 * x.x));
    }
}
template <int R, int J, class MT> __device__ __forceinline__ double rm1r_dot(const double2 *a, const double2 *f, MT dm)
{
    const double m00 = dm[0].x, m01 = dm[1].x, m10 = dm[2].x, m11 = dm[3].x;
    double s = 0;
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if ((k >> J) & 1) continue;
        const int kk = k | (1 << J);
        const double2 x = a[k], y = a[kk];
        // Re(conj(f_k) (m00 x + m01 y)) + Re(conj(f_kk) (m10 x + m11 y))
        s += m00 * zdotr(f[k], x) + m01 * zdotr(f[k], y) + m10 * zdotr(f[kk], x) + m11 * zdotr(f[kk], y);
    }
    return s;
}

// dense 2x2 on register bit J applied where `on` (a control outside the
// stage, per lane): the product is formed on every lane and kept or dropped,
// the matrix entries themselves stay uniform
template <int R, int J, class MT> __device__ __forceinline__ void rm1_on(double2 *a, MT m, bool on)
{
    const double2 m00 = m[0], m01 = m[1], m10 = m[2], m11 = m[3];
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if ((k >> J) & 1) continue;
        const int kk = k | (1 << J);
        const double2 x = a[k], y = a[kk];
        const double2 nx = zmul2(m00, x, m01, y), ny = zmul2(m10, x, m11, y);
        a[k] = on ? nx : x;
        a[kk] = on ? ny : y;
    }
}

// X on register bit J: the pairs swap (no arithmetic); controlled by
// register bit C, or per lane by `on` (a control outside the stage)
template <int R, int J> __device__ __forceinline__ void rx1(double2 *a)
{
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if ((k >> J) & 1) continue;
        const double2 x = a[k];
        a[k] = a[k | (1 << J)];
        a[k | (1 << J)] = x;
    }
}
template <int R, int J, int C> __device__ __forceinline__ void rx1c(double2 *a)
{
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if (((k >> J) & 1) || !((k >> C) & 1)) continue;
        const double2 x = a[k];
        a[k] = a[k | (1 << J)];
        a[k | (1 << J)] = x;
    }
}
template <int R, int J> __device__ __forceinline__ void rx1_if(double2 *a, bool on)
{
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if ((k >> J) & 1) continue;
        const double2 x = a[k], y = a[k | (1 << J)];
        a[k] = on ? y : x;
        a[k | (1 << J)] = on ? x : y;
    }
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
        a[k] = zmul4(m[0], v00, m[1], v01, m[2], v10, m[3], v11);
        a[k01] = zmul4(m[4], v00, m[5], v01, m[6], v10, m[7], v11);
        a[k10] = zmul4(m[8], v00, m[9], v01, m[10], v10, m[11], v11);
        a[k11] = zmul4(m[12], v00, m[13], v01, m[14], v10, m[15], v11);
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
        s += zdotr(f[k], zmul4(m[0], v00, m[1], v01, m[2], v10, m[3], v11));
        s += zdotr(f[k01], zmul4(m[4], v00, m[5], v01, m[6], v10, m[7], v11));
        s += zdotr(f[k10], zmul4(m[8], v00, m[9], v01, m[10], v10, m[11], v11));
        s += zdotr(f[k11], zmul4(m[12], v00, m[13], v01, m[14], v10, m[15], v11));
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
// rf2 for an op whose structure holds for every parameter value: bit 0 / bit
// 3 of U: the |00> / |11> phase is exactly 1 (left out); RX: the block has
// real diagonal and imaginary off-diagonal entries (fSim)
template <int R, int LO, int HI, int U, bool RX, class MT> __device__ __forceinline__ void rf2x(double2 *a, MT m)
{
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if (((k >> LO) & 1) || ((k >> HI) & 1)) continue;
        const int k10 = k | (1 << LO), k01 = k | (1 << HI), k11 = k10 | k01;
        const double2 x = a[k01], y = a[k10];
        if (!(U & 1)) a[k] = zmul(m[0], a[k]);
        if (RX) {
            const double b00 = m[1].x, b01 = m[2].y, b10 = m[3].y, b11 = m[4].x;
            a[k01] = make_double2(fma(b00, x.x, -b01 * y.y), fma(b00, x.y, b01 * y.x));
            a[k10] = make_double2(fma(b11, y.x, -b10 * x.y), fma(b11, y.y, b10 * x.x));
        } else {
            a[k01] = zmul2(m[1], x, m[2], y);
            a[k10] = zmul2(m[3], x, m[4], y);
        }
        if (!(U & 8)) a[k11] = zmul(m[5], a[k11]);
    }
}
// rf2 for an op whose (|01>, |10>) block is -i SWAP (kHintSwap: fSim(pi/2,
// phi)): the pair trades places with a factor -i, (x, y) -> (y, -x), and only
// the |00> / |11> phases that are not exactly 1 (U as in rf2x) are multiplied
template <int R, int LO, int HI, int U, class MT> __device__ __forceinline__ void rf2s(double2 *a, MT m)
{
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if (((k >> LO) & 1) || ((k >> HI) & 1)) continue;
        const int k10 = k | (1 << LO), k01 = k | (1 << HI), k11 = k10 | k01;
        const double2 x = a[k01], y = a[k10];
        a[k01] = make_double2(y.y, -y.x);
        a[k10] = make_double2(x.y, -x.x);
        if (!(U & 1)) a[k] = zmul(m[0], a[k]);
        if (!(U & 8)) a[k11] = zmul(m[5], a[k11]);
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
        a[k] = zmul2(ca, v00, bs, v11);
        a[k11] = zmul2(ca, v11, bs, v00);
        a[kL] = zmul2(ca, vL, cb, vH);
        a[kH] = zmul2(ca, vH, cb, vL);
    }
}
// rp2 with a real and b imaginary (XX^t without its global phase, and its
// products): half the arithmetic
template <int R, int LO, int HI> __device__ __forceinline__ void rp2x(double2 *a, double2 ca, double2 cb, double sg)
{
    const double p = ca.x, q = cb.y, qs = sg * cb.y;
#pragma unroll
    for (int k = 0; k < (1 << R); k++) {
        if (((k >> LO) & 1) || ((k >> HI) & 1)) continue;
        const int kL = k | (1 << LO), kH = k | (1 << HI), k11 = kL | kH;
        const double2 v00 = a[k], vL = a[kL], vH = a[kH], v11 = a[k11];
        a[k] = make_double2(fma(p, v00.x, -qs * v11.y), fma(p, v00.y, qs * v11.x));
        a[k11] = make_double2(fma(p, v11.x, -qs * v00.y), fma(p, v11.y, qs * v00.x));
        a[kL] = make_double2(fma(p, vL.x, -q * vH.y), fma(p, vL.y, q * vH.x));
        a[kH] = make_double2(fma(p, vH.x, -q * vL.y), fma(p, vH.y, q * vL.x));
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
        s += zdotr(f[k], zmul2(ca, a[k], bs, a[k11]));
        s += zdotr(f[k11], zmul2(ca, a[k11], bs, a[k]));
        s += zdotr(f[kL], zmul2(ca, a[kL], cb, a[kH]));
        s += zdotr(f[kH], zmul2(ca, a[kH], cb, a[kL]));
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
        if (op.hint & kHintX) {
            // a constant X (CNOT's target block): the pairs swap, no gradient
            if (!op.ctrl) {
                TQ_BIT_SWITCH(R, op.s0, ({ rx1<R, j_>(a); rx1<R, j_>(f); }))
            } else if (op.s1 != kFixed) {
                TQ_ORDERED_SWITCH(R, op.s0, op.s1, ({ rx1c<R, j_, c_>(a); rx1c<R, j_, c_>(f); }))
            } else {
                const bool on = ctrl_on(op, base, fb);
                TQ_BIT_SWITCH(R, op.s0, ({ rx1_if<R, j_>(a, on); rx1_if<R, j_>(f, on); }))
            }
        } else if (!op.ctrl && (op.hint & kHintReal)) {
            TQ_BIT_SWITCH(R, op.s0, ({
                rm1r<R, j_>(a, m);
                if (op.ngrad > 0) g0 += rm1r_dot<R, j_>(a, f, d0);
                if (op.ngrad > 1) g1 += rm1r_dot<R, j_>(a, f, d1);
                rm1r<R, j_>(f, m);
            }))
        } else if (!op.ctrl) {
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
template <int R, class MT> __device__ __forceinline__ void rdense(double2 *a, MT S)
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

// ------------------------------------------- resident circuit parts
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

// Stage the matrices [begin, end) of a row block into LDS.
__device__ __forceinline__ void stage_mats(double2 *dst, const double2 *row_block, int begin, int end)
{
    for (int i = begin + (int)threadIdx.x; i < end; i += blockDim.x) dst[i - begin] = row_block[i];
}

// ---------------------------------------------------------- tile pass parts
// The parts of a forward or reverse tile pass around its register stages
// (which the generic kernels loop over and a specialised kernel spells out).
struct PassCtx {
    float2 *lds;        // the tile
    double2 *lm;        // the pass's matrices
    double2 *p1, *p2;   // product-state factors over the tile's low / high halves
    uint64_t *hi_off;
    float2 *st;         // the row's state
    int row, w, a1;
};

__device__ __forceinline__ PassCtx pass_setup(const PassArgs &a, unsigned char *smem)
{
    const TileGeom &g = a.g;
    const int t = g.t;
    PassCtx c;
    c.lds = reinterpret_cast<float2 *>(smem);
    c.hi_off = reinterpret_cast<uint64_t *>(smem + sizeof(float2) * (1 << t));
    c.lm = reinterpret_cast<double2 *>(c.hi_off + (1 << g.h));
    c.p1 = c.lm + (a.mat_end - a.mat_begin);
    c.a1 = t / 2;
    c.p2 = c.p1 + (1 << c.a1);
    c.row = blockIdx.x / a.wg_per_row;
    c.w = blockIdx.x % a.wg_per_row;
    c.st = a.state + (int64_t)cget(a.rows, c.row) * a.row_stride;
    build_hi_off(g, c.hi_off);
    stage_mats(c.lm, a.mats + (int64_t)c.row * a.mat_stride, a.mat_begin, a.mat_end);
    __syncthreads();
    if (a.product_init) {
        // per-qubit product-state vectors: column 0 of each init matrix
        const double2 *M = c.lm;  // offsets relative to mat_begin
        for (int j = threadIdx.x; j < (1 << c.a1) + (1 << (t - c.a1)); j += blockDim.x) {
            const bool first = j < (1 << c.a1);
            const int k0 = first ? 0 : c.a1, k1 = first ? c.a1 : t;
            const int v = first ? j : j - (1 << c.a1);
            double2 acc = make_double2(1.0, 0.0);
            for (int k = k0; k < k1; k++) {
                int pos = k < g.c ? k : g.hb[k - g.c];
                int q = g.n - 1 - pos;
                const double2 *im = M + (a.init_mat[q] - a.mat_begin);
                acc = zmul(acc, ((v >> (k - k0)) & 1) ? im[2] : im[0]);
            }
            if (first) c.p1[v] = acc;
            else c.p2[v] = acc;
        }
    }
    __syncthreads();
    return c;
}

// the tile with fixed bits fb into LDS (generated product state in the first pass)
__device__ __forceinline__ void pass_load(const PassArgs &a, const PassCtx &c, uint64_t fb)
{
    const TileGeom &g = a.g;
    const int T = 1 << g.t;
    if (a.product_init) {
        const double2 *M = c.lm;
        double2 f = make_double2(1.0, 0.0);
        for (uint64_t fm = g.fixed_mask; fm; fm &= fm - 1) {
            int pos = __ffsll((unsigned long long)fm) - 1;
            const double2 *im = M + (a.init_mat[g.n - 1 - pos] - a.mat_begin);
            f = zmul(f, ((fb >> pos) & 1) ? im[2] : im[0]);
        }
        for (int l = threadIdx.x; l < T; l += blockDim.x)
            c.lds[sw(l)] = down2(zmul(f, zmul(c.p1[l & ((1 << c.a1) - 1)], c.p2[l >> c.a1])));
    } else {
        TileCtx tc{c.hi_off, (1u << g.c) - 1, g.c};
        tile_copy<true>(tc, c.lds, c.st, fb, T);
    }
}

__device__ __forceinline__ void pass_store(const PassArgs &a, const PassCtx &c, uint64_t fb)
{
    TileCtx tc{c.hi_off, (1u << a.g.c) - 1, a.g.c};
    tile_copy<false>(tc, c.lds, c.st, fb, 1 << a.g.t);
}

struct RevCtx {
    float2 *lp, *lf;    // psi and phi tiles
    uint64_t *hi_off;
    double2 *lm;        // the pass's matrices
    double *acc;        // [4 waves][gcount] gradient partials
    float2 *sp, *sf;    // the row's psi and phi
    int row, w;
};

__device__ __forceinline__ RevCtx rev_setup(const RevArgs &a, unsigned char *smem)
{
    const TileGeom &g = a.g;
    const uint32_t T = 1u << g.t;
    RevCtx c;
    c.lp = reinterpret_cast<float2 *>(smem);
    c.lf = c.lp + T;
    c.hi_off = reinterpret_cast<uint64_t *>(c.lf + T);
    c.lm = reinterpret_cast<double2 *>(c.hi_off + (1 << g.h));
    c.acc = reinterpret_cast<double *>(c.lm + (a.mat_end - a.mat_begin));
    c.row = blockIdx.x / a.wg_per_row;
    c.w = blockIdx.x % a.wg_per_row;
    const int b = cget(a.rows, c.row);
    c.sp = a.psi + (int64_t)b * a.row_stride;
    c.sf = a.phi + (int64_t)b * a.row_stride;
    build_hi_off(g, c.hi_off);
    stage_mats(c.lm, a.mats + (int64_t)c.row * a.mat_stride, a.mat_begin, a.mat_end);
    for (int j = threadIdx.x; j < 4 * a.gcount; j += blockDim.x) c.acc[j] = 0;
    __syncthreads();
    return c;
}

__device__ __forceinline__ void rev_load(const RevArgs &a, const RevCtx &c, uint64_t fb)
{
    TileCtx tc{c.hi_off, (1u << a.g.c) - 1, a.g.c};
    tile_copy<true>(tc, c.lp, c.sp, fb, 1 << a.g.t);
    tile_copy<true>(tc, c.lf, c.sf, fb, 1 << a.g.t);
}

__device__ __forceinline__ void rev_store(const RevArgs &a, const RevCtx &c, uint64_t fb)
{
    if (!a.store) return;
    TileCtx tc{c.hi_off, (1u << a.g.c) - 1, a.g.c};
    tile_copy<false>(tc, c.lp, c.sp, fb, 1 << a.g.t);
    tile_copy<false>(tc, c.lf, c.sf, fb, 1 << a.g.t);
}

// the workgroup's gradient partials, waves summed in a fixed order
__device__ __forceinline__ void rev_finish(const RevArgs &a, const RevCtx &c)
{
    double *out = a.gpart + ((int64_t)c.row * a.wg_per_row + c.w) * a.n_gslots + a.gbase;
    for (int j = threadIdx.x; j < a.gcount; j += blockDim.x)
        out[j] = ((c.acc[j] + c.acc[a.gcount + j]) + c.acc[2 * a.gcount + j]) + c.acc[3 * a.gcount + j];
}

} // namespace tq
