// tq_internal.h -- data structures shared by the host planner and the HIP
// kernels of libtq.  Nothing here is part of the public ABI.
#pragma once
#ifdef __HIPCC_RTC__
// the run-time compiler brings its own fixed-width integer types
using __hip_internal::int32_t;
using __hip_internal::int64_t;
using __hip_internal::uint16_t;
using __hip_internal::uint32_t;
using __hip_internal::uint64_t;
using __hip_internal::uint8_t;
#else
#include <cstdint>
#endif

namespace tq {

// Opcodes of the program blob (the public list is in include/tq.h).
enum Opcode : uint16_t {
    OP_H = 1, OP_X, OP_Y, OP_Z, OP_RX, OP_RY, OP_RZ, OP_XPOW, OP_YPOW, OP_ZPOW,
    OP_CZ, OP_CNOT, OP_CZPOW, OP_CNOTPOW, OP_XXPOW, OP_YYPOW, OP_ZZPOW, OP_RZZ,
    OP_SQRTX, OP_SQRTY, OP_SQRTW, OP_FSIM, OP_MATRIX1, OP_MATRIX2, OP_SWAP,
    // Pauli channel on one qubit (X, Y, Z with the constant probabilities of
    // its three parameters): each row, one trajectory, draws its Pauli
    OP_PCHAN = 27,
    OP_COUNT
};
// exp(-i eta P) of a Pauli string: a blob opcode only, lowered to the gates
// above when a program is parsed
constexpr uint16_t OP_PAULIEXP = 26;

constexpr int kMaxQubits = 32;
constexpr int kThreads = 256;  // threads per workgroup of every tile kernel
constexpr uint8_t kFixed = 0xFF;  // "bit not in the tile" marker
constexpr int kMaxGradPerPass = 512;  // gradient slots one reverse pass accumulates
constexpr int kMaxPassMat = 2048;     // matrix entries (complex128) one pass stages in LDS

// One gate of a structure, as the device matrix builder reads it.
struct GateDev {
    uint16_t op;
    uint8_t nq, np;
    int32_t slot0;     // first of its np parameter slots
    int32_t explicit_; // index of its explicit matrix (MATRIX1/2) or -1
    int32_t chan;      // OP_PCHAN: its ordinal among the circuit's channels, else -1
};

// How a matrix is rendered by the builder.
enum Form : uint8_t {
    FORM_FULL = 0,   // 2x2 for 1q gates, 4x4 for 2q gates
    FORM_CBLOCK = 1, // 2x2 target block of a controlled gate (CNOT, CNOTPOW)
};

// A member of a fused product: gate index, and for a 2q gate inside a 2q
// product whether its qubit order is reversed relative to the product's.
struct Member {
    int32_t gate;
    uint8_t swapped;
    uint8_t form;
    uint8_t pad[2];
};

// One term of a row's global phase (the phases the gate matrices leave out):
// c * eta(slot), or the constant c when slot < 0.
struct PhaseTerm {
    int32_t slot;
    int32_t pad;
    double c;
};

// Build tasks of the matrix builder; each writes one matrix per batch row.
enum TaskKind : uint8_t {
    BT_PRODUCT = 0, // product of members (last member applied last)
    BT_DAGGER = 1,  // conjugate transpose of a single member
    BT_DERIV = 2,   // derivative of a single member w.r.t. parameter `which`
};

struct BuildTask {
    uint8_t kind;
    uint8_t dim;    // 2 or 4
    uint8_t diag;   // storage: 0 dense, 1 diagonal (dim entries), 2 / 3 the pair (a, b) of
                    // a I + b XX / a I + b YY, 4 the six entries of an excitation-preserving 4x4
    uint8_t which;  // BT_DERIV parameter index
    int32_t out;    // offset (complex entries) in the row's matrix block
    int32_t mem_begin, mem_count;
};

// Kinds of ops a tile pass applies.
enum OpKind : uint8_t {
    K_M1 = 1, // dense 2x2 on local bit q0; optional control qubit q1
    K_M2 = 2, // dense 4x4 on local bits (q0 = first qubit, q1 = second)
    K_D1 = 3, // diagonal on q0 (local or fixed)
    K_D2 = 4, // diagonal on (q0, q1), entry index 2*bit(q0) + bit(q1)
    K_P2 = 5, // a I + b P on local bits (q0, q1) with P = XX (ptype 1) or YY (ptype 2)
    K_F2 = 6, // excitation preserving on local bits (q0, q1): phase on |00>, 2x2 block on
              // (|01>, |10>), phase on |11> (fSim, SWAP and their products with diagonals)
};

constexpr uint8_t kHintX = 16;
constexpr uint8_t kHintReal = 32;  // K_M1: the matrix and its derivatives are real
// K_M1: real diagonal and imaginary off-diagonal entries (RX and its products;
// so are the derivatives); K_F2: the (|01>, |10>) block has that form (fSim);
// K_P2: a real and b imaginary
constexpr uint8_t kHintRX = 64;
// K_F2, forward ops of generated kernels: the (|01>, |10>) block is -i SWAP
// (fSim(theta, phi) with a constant theta whose cosine is below 1e-15 and
// sine within 1e-15 of 1 in every row: its diagonal entries, ~6e-17, are
// taken as 0 and the off-diagonal ones as exactly -i)
constexpr uint8_t kHintSwap = 128;
struct PassOp {
    uint8_t kind;
    uint8_t l0, l1;   // local bit of q0 / q1 in the tile, kFixed if outside
    uint8_t p0, p1;   // global bit position of q0 / q1
    uint8_t ctrl;     // K_M1: 1 if q1 is a control qubit
    uint8_t cval;     // K_M1: the control value that enables the op
    uint8_t ngrad;    // reverse ops: symbolic parameters (0..2)
    uint8_t ptype;    // K_P2: 1 = XX, 2 = YY
    uint8_t s0, s1;   // register index of q0 / q1 within the op's stage, kFixed if not in it
    uint8_t hint;     // structure every parameter value keeps: K_D1 / K_D2 bit k (k < 4): diagonal
                      // entry k of the matrix is exactly 1 (and of dW/deta exactly 0); K_M1
                      // kHintX: the matrix is exactly X (a swap); kHintReal: it is real;
                      // kHintRX (K_M1, K_F2, K_P2) as above; K_F2 bit 0 / bit 3: the phase on
                      // |00> / |11> is exactly 1
    int32_t mat;      // offset of the op's matrix (forward) or W^dagger (reverse)
    int32_t dmat[2];  // reverse: offsets of dW/deta_j
    int32_t gslot[2]; // reverse: gradient slot ids
};

// A stage: consecutive ops of a pass whose dense qubits lie in a set R of at
// most kStageBits tile bits.  Each thread holds the 2^r amplitudes of one
// "item" (a fixed assignment of the tile bits outside R) in registers while
// the stage's ops run, so the stage costs one LDS round trip.
constexpr int kStageBitsFwd = 3;
constexpr int kStageBitsRev = 3;
constexpr int kRevDense2Bits = 2;  // reverse stages holding a dense 4x4 or fSim-type op
constexpr int kStageBitsRevResident = 2;  // circuits small enough for the resident kernel
// Gradient parameters of one reverse stage: each thread keeps their partial
// sums in registers over the stage's items.
constexpr int kMaxStageGrads = 8;
struct Stage {
    uint8_t r;        // register bits
    uint8_t bits[4];  // their tile-local positions, ascending
    uint8_t dense;    // 1: the stage's ops are applied as one 2^r x 2^r matrix
    uint8_t pad[2];
    int32_t op_begin, op_end;  // ops, as indices into the group's op array
    int32_t mat;      // dense: offset of the stage matrix (row major) in the row block
};

// Tile geometry of a pass: t local bits = `c` low bits + high bits hb[].
struct TileGeom {
    int32_t n, t, c, h;
    uint64_t fixed_mask; // global bits (< n) outside the tile
    uint8_t hb[kMaxQubits];
};

// A Pauli term with masks in global index bits and in tile-local bits.
struct TermDev {
    uint64_t x, z;      // global masks
    uint64_t xout;      // bits of x outside the tile
    uint32_t xl, zl;    // local masks
    int32_t k;          // observable index
    int32_t ny;         // number of Y factors (mod 4 used)
    double coeff;
};

// Pauli sums in the form the tile kernel evaluates them.  With l a tile-local
// index, the thread layout l = tid + 256 r splits l into its low 8 bits (the
// thread) and the bits above (the thread's register r).  A term
// c i^{ny} X^x Z^z acts on a tile with fixed bits fb as
//     (P psi)_l = c' chi_zF(fb) chi_zlo(tid) chi_u(r) psi_{l ^ xT} (tile fb ^ xF),
// chi_m(v) = (-1)^{|m & v|}, where c' = c i^{ny} chi_z(x) is real or purely
// imaginary.  Terms are grouped by observable chunk, then by the out-of-tile
// part xF of x (one partner tile per group), then by (xT, observable), then
// by u, so that the per-amplitude work is one partner read per x group.
constexpr int kPauliChunk = 4;  // observables accumulated together
struct PTerm {
    uint64_t zF;     // z outside the tile (global bits)
    uint32_t zlo;    // z on tile bits 0..7
    uint32_t im;     // 1: c' is imaginary (value in c)
    double c;        // real or imaginary part of c'
};
struct PUSub {       // terms sharing u = z on tile bits 8..t-1
    uint32_t u;
    int32_t t_begin, t_end;
    int32_t pad;
};
struct PXGroup {     // terms of one observable sharing x
    uint32_t xT;     // x on the tile bits
    int32_t kk;      // observable within the chunk
    int32_t u_begin, u_end;
    uint32_t flags;  // 1: some c' real, 2: some c' imaginary
    int32_t pad;
};
struct PXfGroup {    // x groups sharing the partner tile fb ^ xF
    uint64_t xF;
    int32_t x_begin, x_end;
};
struct PChunk {      // observables [k0, k0 + nk), nk <= kPauliChunk
    int32_t k0, nk;
    int32_t xf_begin, xf_end;
};

// Diagonal (Z-only) Pauli sums over whole states, read straight from HBM.
// A state is cut into blocks of 2^12 amplitudes; thread tid of a block holds
// the 16 amplitudes 512 j + 2 tid + e (j < 8, e < 2).  With r = e + 2 j the
// register index, a term c Z^z splits z into zB (block bits 12..n-1), zT
// (bits 1..8, the thread) and v (bit 0 and bits 9..11, the register):
//     <Z^z> = sum_blk chi_zB(blk) sum_tid chi_zT(tid) W_v(blk, tid),
//     W_v = sum_r chi_v(r) |psi|^2,
// so each thread needs the Walsh transform W of its 16 probabilities and one
// accumulator per class of terms sharing (observable, v, zT); the sign of
// the block is folded into a per-block class weight
// D(blk) = sum_{t in class} c_t chi_zB_t(blk).
constexpr int kDiagBlockBits = 12;
constexpr int kDiagClassMax = 32;   // classes accumulated in one sweep
constexpr int kDiagRefill = 64;     // blocks whose class weights are staged at once
struct DTerm {
    uint64_t zB;     // z on the block bits, shifted down by kDiagBlockBits
    double c;
};
struct DClass {
    int32_t k;       // observable
    uint32_t v;      // register mask (bit 0: index bit 0; bits 1..3: index bits 9..11)
    uint32_t zT;     // thread mask (index bits 1..8)
    int32_t t_begin, t_end;
    int32_t pad;
};
struct DChunk {      // classes swept together, observables k_lo..k_hi
    int32_t c_begin, c_end;
    int32_t k_lo, k_hi;
};

} // namespace tq
