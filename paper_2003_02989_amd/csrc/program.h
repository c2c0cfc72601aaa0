// program.h -- host-side program representation: parsed circuits, structure
// groups (circuits of the batch that share gates and symbol wiring) and the
// pass plans the kernels execute.
#pragma once
#include <algorithm>
#include <memory>
#include <string>
#include <vector>

#include "tq_internal.h"

namespace tq {

struct Error {
    int status;
    std::string msg;
};

struct Options {
    int tile = 12;    // forward tile bits
    int low = 6;      // contiguous low bits per tile
    bool fuse = true;
    int max_pass_gates = 0;  // 0: no limit
    bool specialize = false; // kernels compiled per circuit structure at run time
};

struct HGate {
    uint16_t op;
    uint8_t nq, np;
    uint32_t q[2];
    int32_t sym[3];
    double scale[3], offset[3];
    double mat[32];
    // the blob gate it comes from (its index in the circuit and opcode) and,
    // for gates lowered from a Pauli-string exponential, the factor its
    // parameter carries (parameter = mult x the exponential's eta)
    int32_t origin;
    uint16_t blob_op;
    double mult;
};

// A symbolic parameter of a blob gate (what the parameter-shift rule shifts
// one at a time), in gate and parameter order.  The gates lowered from a
// Pauli-string exponential carry its parameter in one slot (two for the
// global phase of weight zero), each as mult x eta.
struct Occurrence {
    int32_t slot[2];   // the parameter slots it drives (slot[1] = -1: one)
    double mult[2];
    int32_t sym;
    uint16_t blob_op;  // opcode of the blob gate
    uint8_t param;     // its parameter index in the blob gate
};

// The two-term shift rule of parameter `param` of blob opcode `op` (Sec.
// "Parameter shift methods", eq. parshift_grad): when the parameter eta
// enters as exp(-i eta G) and G has two distinct eigenvalues a gap r apart,
// every expectation is c0 + c1 cos(r eta) + c2 sin(r eta), and
// df/deta = (r/2) (f(eta + pi/(2r)) - f(eta - pi/(2r))).  Gives delta =
// pi/(2r) and factor = r/2; false for a parameter without such a rule
// (fSim's theta: three eigenvalues).
bool shift_rule(int op, int param, double *delta, double *factor);

struct HCircuit {
    int n = 0;  // (gates live in the circuit's structure group)
};

struct Pass {
    TileGeom geom;
    std::vector<PassOp> ops;
    bool product_init = false;
    int32_t mat_begin = 0, mat_end = 0;  // the pass's matrices in the row block
    int32_t op_offset = 0;               // index of the pass's first op in the group's op array
    std::vector<Stage> stages;           // op indices relative to the group's op array
};

// Build-task ranges of a group: [begin, end) into Group::tasks.
struct TaskRange {
    int begin = 0, end = 0;
};

struct Group {
    int n = 0;
    std::vector<int32_t> rows;  // batch indices of the circuits in this group
    std::vector<GateDev> gates;
    std::vector<int32_t> gate_q0, gate_q1;
    int n_slots = 0;
    std::vector<int32_t> slot_sym;              // [n_slots]
    std::vector<double> slot_scale, slot_off;   // [rows or 1][n_slots]
    bool uniform_slots = true;
    std::vector<double> explicit_mats;          // [n_explicit][32]

    // plan
    std::vector<BuildTask> tasks;
    std::vector<Member> members;
    TaskRange fwd_tasks, rev_tasks;
    int32_t mat_block = 0;                      // complex entries per row
    std::vector<Pass> fwd;
    int32_t init_mat[kMaxQubits];               // per qubit: 2x2 product-init matrix
    std::vector<Pass> rev;
    int n_gslots = 0;
    std::vector<int32_t> gslot_slot;            // gradient slot -> parameter slot
    std::vector<int32_t> sym_gslot_begin;       // [S+1] CSR symbol -> gradient slots
    std::vector<int32_t> sym_gslots;
    int32_t fwd_mat_end = 0;                    // forward matrices (with the product init) end here
    std::vector<std::pair<int, int>> dense_stages;  // (forward pass, stage) with a stage matrix
    std::vector<PhaseTerm> phase_terms;         // the row's global phase, linear in the parameters
    std::vector<Occurrence> occurrences;        // symbolic blob parameters, in gate and parameter order
};

// Per-op dispatch overhead of the register ops, in fp64-instruction
// equivalents per amplitude (measured: ~6 for 2x2 ops at three register bits).
constexpr int kOpDispatchCost = 6;
// The same for kernels generated for the circuit structure, whose ops are
// straight-line code (no table reads or dispatch; a register move or two).
constexpr int kOpDispatchCostSpec = 0;
// One register stage's LDS round trip in the same units (measured: ~0.29 ms
// per stage of a 2^30-amplitude pass).
constexpr int kStageCost = 11;

// Generators of the parameterised gates.  Every such gate is, as a function
// of one of its parameters eta, W(eta) = exp(-i eta G) times factors that
// commute with G and do not depend on eta, so dW/deta = -i G W and the
// adjoint term Re<phi| dW |psi_before> equals Im<phi| G |psi_after>
// (Sec. "Adjoint Gradient Backpropagation in Simulations").  G is given as
// real-weighted Pauli strings c i^ny X^x Z^z on the op's qubits (bit 0 of x
// and z: the op's q0, bit 1: its q1).
struct GenTerm {
    uint8_t x, z, ny;
    double c;
};
// The generator of parameter j of reverse op `op` (a single gate); false when
// the gate has none of the listed forms.
bool op_generator(const Group &g, const PassOp &op, int j, std::vector<GenTerm> *terms);

// Register bits of reverse stages.  Circuits small enough for the resident
// kernel keep kStageBitsRevResident (the width the precompiled resident kernel
// is compiled for), except states of at most kWideRevQubits qubits whose
// kernel is generated per structure: there a workgroup of one thread per
// three-bit item runs kStageBitsRev-bit stages (half the LDS round trips).
constexpr int kWideRevQubits = 10;
inline int rev_stage_bits(int n, const Options &opt)
{
    if (n > std::min(opt.tile, 12)) return kStageBitsRev;
    return opt.specialize && n <= kWideRevQubits ? kStageBitsRev : kStageBitsRevResident;
}

struct ProgramData {
    int B = 0, S = 0, nmax = 0;
    Options opt;
    std::vector<HCircuit> circuits;
    std::vector<std::unique_ptr<Group>> groups;
};

struct HTerm {
    double coeff;
    std::vector<std::pair<uint32_t, uint8_t>> factors;  // (qubit, pauli 1..3)
};

struct ObsData {
    int B = 0, K = 0;
    std::vector<std::vector<HTerm>> sums;  // [B*K]
    uint64_t id = 0;
};

// The global phase (radians) the device builder leaves out of the matrix of
// gate `op` with first parameter eta: the full gate matrix is e^{i phase}
// times the one built.
double gate_left_out_phase(int op, double eta);

std::unique_ptr<ProgramData> parse_program(const void *blob, size_t nbytes, const Options &opt);
std::unique_ptr<ObsData> parse_observables(const void *blob, size_t nbytes);

// Tile geometry for expectation-type kernels: low bits plus the bits most
// often flipped by the terms' X/Y factors.
TileGeom expectation_geometry(int n, int t, int c, const std::vector<uint64_t> &xmasks);

// Term tables of the tile Pauli kernel for the rows of one structure group
// (terms given with global masks x, z, their Y count, observable and
// coefficient).  Rows with identical term lists may share one table
// (`uniform`).  Every row gets ceil(K / kPauliChunk) chunks.
struct PauliTables {
    TileGeom geom;
    bool partner = false;  // some term flips a bit outside the tile
    std::vector<PChunk> chunks;
    std::vector<int32_t> row_begin, row_count;
    std::vector<PXfGroup> xfg;
    std::vector<PXGroup> xg;
    std::vector<PUSub> us;
    std::vector<PTerm> terms;
};
PauliTables pauli_tables(int n, int t, int c, int K, const std::vector<std::vector<TermDev>> &per_row, bool uniform);

// Passes of the Pauli kernel specialised for one observable set (the same
// terms on every row): each pass's tile holds the X bits of all its terms, so
// that every partner amplitude is in the tile and the state is read once per
// pass.  Terms are given with global masks.
struct SpecTerm {
    int k;            // observable
    uint64_t x, z;
    int ny;           // Y factors
    double coeff;
};
struct PauliPass {
    TileGeom geom;
    std::vector<SpecTerm> terms;
};
// Plans passes over tiles of t bits (c low bits); false when some term flips
// more bits above the low ones than a tile holds.
bool pauli_spec_plan(int n, int t, int c, const std::vector<TermDev> &terms, std::vector<PauliPass> *passes);

// Tables of the diagonal (Z-only) Pauli kernel: every term of every row must
// have x = 0 and the states at least kDiagBlockBits qubits.
struct DiagTables {
    std::vector<DChunk> chunks;
    std::vector<int32_t> row_begin, row_count;
    std::vector<DClass> classes;
    std::vector<DTerm> terms;
    int amax = 0;  // largest class count of a chunk
};
DiagTables diag_tables(const std::vector<std::vector<TermDev>> &per_row, bool uniform);

} // namespace tq
