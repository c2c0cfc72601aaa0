// kernel_args.h -- argument blocks of the libtq kernels (plain structs that
// the host fills and the kernels take by value).
#pragma once
#ifndef __HIPCC_RTC__
#include <hip/hip_runtime.h>
#endif

#include "tq_internal.h"

namespace tq {

constexpr int kMaxLevels = 8;    // sampler levels (64-ary), enough for 2^48 amplitudes

// The parameter moves of one derived row of the batched shift rules: the
// parameter-shift rule moves eta of one or two slots (a Pauli-string
// exponential's lowered gates move together), central differences move one
// symbol value.
struct ShiftDev {
    int32_t slot[2];   // slots whose eta moves by delta (-1: none)
    int32_t sym;       // symbol whose value moves by dtheta x eps (-1: none)
    int32_t pad;
    double delta[2];
    double dtheta;
};

struct BuildArgs {
    const BuildTask *tasks;
    int task_begin, task_end;
    const Member *members;
    const GateDev *gates;
    const int32_t *slot_sym;
    const double *slot_scale, *slot_off;
    int uniform, n_slots;
    const double *explicit_mats;
    const float *theta;
    int S;
    const int32_t *rows;
    double2 *mats;
    int64_t mat_stride;
    // the task writing this matrix offset (the first qubit's product-init
    // matrix; the first task of the range) also multiplies it by the row's
    // global phase, the sum of the phases the gate matrices leave out; -1: none
    int32_t phase_out;
    int32_t n_phase;
    const PhaseTerm *phase_terms;
    // seed of the channels' per-row Kraus draws
    uint64_t noise_seed;
    // derived rows of the batched shift rules (x_period = 0: the rows
    // themselves): launch row r is row L = x_begin + r of the group's
    // expansion, a copy of group row L / x_period with the parameter moves of
    // x_shift[L % x_period]
    int64_t x_begin;
    int32_t x_period;
    const ShiftDev *x_shift;
    double x_eps;            // symbol moves are dtheta x x_eps
    // derived rows built from their source row's block: the block's first
    // x_copy entries are copied from x_src (the source rows' blocks), then
    // only the tasks task_list[list_begin[m] .. list_begin[m + 1]) of the
    // row's move m are built again.  When the row carries a global phase,
    // either the list starts with the task of phase_out (its members have a
    // moved parameter), which takes the derived row's whole phase, or the
    // copied phase_out matrix, holding the source row's phase, is multiplied
    // by the change of the phase terms phase_list[phase_begin[m] ..
    // phase_begin[m + 1]) (the terms of a moved parameter); phase_full[m]
    // says which
    const double2 *x_src;
    int32_t x_copy;
    const int32_t *list_begin, *task_list;
    const int32_t *phase_full, *phase_begin, *phase_list;
};

struct StageBuildArgs {
    const Stage *stages;   // the group's forward stages
    const int32_t *list;   // indices of the dense ones
    int nlist;
    const PassOp *ops;     // the group's forward ops
    double2 *mats;
    int64_t mat_stride;
};

struct PassArgs {
    float2 *state;
    int64_t row_stride;
    const int32_t *rows;
    const double2 *mats;
    int64_t mat_stride;
    const PassOp *ops;     // the group's forward ops (stages index them)
    const Stage *stages;   // this pass's stages
    int nstages;
    TileGeom g;
    int tiles_log2;
    int wg_per_row;
    int product_init;
    int32_t init_mat[kMaxQubits];
    int mat_begin, mat_end;  // the pass's matrices, staged in LDS
};

struct PauliArgs {
    const float2 *psi;
    float2 *phi;             // NULL: expectations only
    int phi_accumulate;      // add into phi instead of overwriting it
    int64_t row_stride;
    const int32_t *rows;     // state rows
    const int32_t *brows;    // batch index of each row (upstream)
    const PChunk *chunks;
    const int32_t *row_chunk_begin, *row_chunk_count;
    const PXfGroup *xfg;
    const PXGroup *xg;
    const PUSub *us;
    const PTerm *terms;
    const float *upstream;   // [B, K] (phi only)
    int K;                   // observables per row (upstream stride)
    int k_begin, k_count;    // observables of this launch
    TileGeom g;
    int tiles_log2, wg_per_row;
    double *partial;         // [nrows][wg_per_row][k_count]
};

struct DiagArgs {
    const float2 *psi;
    int64_t row_stride;
    const int32_t *rows;     // state rows
    const DChunk *chunks;
    const int32_t *row_chunk_begin, *row_chunk_count;
    const DClass *classes;
    const DTerm *terms;
    int k_begin, k_count;    // observables of this launch
    int blocks_log2, wg_per_row;
    double *partial;         // [nrows][wg_per_row][k_count]
};

// A pass of the Pauli kernel specialised for one observable set.
struct PauliSpecArgs {
    const float2 *psi;
    int64_t row_stride;
    const int32_t *rows;     // state rows
    TileGeom g;              // the pass's tile
    int wg_per_row;
    int npass, pass;         // partial slots: [nrows][npass][wg_per_row][k_count]
    int k_count;
    double *partial;
};

// phi = g H psi for a single observable H (the same on every row) and its
// expectation, pass by pass over tiles that hold the X bits of the pass's
// terms (kernels tq_hphi_<pass> generated for the observable).
struct HPhiArgs {
    const float2 *psi;
    float2 *phi;             // written by pass 0, accumulated by the others
    int64_t row_stride;
    const int32_t *rows;     // state rows
    const int32_t *brows;    // batch index of each row (upstream)
    const float *upstream;   // [B][K]: g = upstream[b][0]
    int K;
    TileGeom g;              // the pass's tile
    int wg_per_row;
    int npass, pass;         // partial slots: [nrows][npass][wg_per_row]
    double *partial;
};

struct PauliReduceArgs {
    const int32_t *rows;     // batch index of each row
    const double *partial;
    int wg_per_row, K, k_begin, k_count;
    float *out;
};

struct RevArgs {
    float2 *psi, *phi;
    int64_t row_stride;
    const int32_t *rows;
    const double2 *mats;
    int64_t mat_stride;
    const PassOp *ops;     // the group's reverse ops
    const Stage *stages;   // this pass's stages
    int nstages;
    TileGeom g;
    int tiles_log2, wg_per_row;
    int store;
    double *gpart;  // [nrows][wg_per_row][n_gslots]
    int n_gslots, gbase, gcount;
    int mat_begin, mat_end;
};

struct ResArgs {
    const double2 *mats;  // row blocks built by k_build_mats
    int64_t mat_stride;
    const double *slot_scale;
    int uniform, n_slots;
    int S;
    const int32_t *rows;  // batch index of each row
    int n;
    const PassOp *fops;
    const Stage *fstages;
    int nfstages;
    int32_t init_mat[kMaxQubits];
    // optional state output
    float2 *state_out;
    int64_t out_stride;
    const int32_t *out_rows;
    // optional expectations
    const TermDev *terms;
    const int32_t *row_term_begin, *row_term_count;
    int K;
    float *exp_out;
    int nacc, gacc;  // accumulators: [0, gacc) terms, [gacc, gacc + n_gslots) gradients
    // optional adjoint
    const PassOp *rops;
    const Stage *rstages;
    int nrstages;
    const float *upstream;
    const int32_t *sym_begin, *sym_gslots, *gslot_slot;
    float *grad;
};

struct GradReduceArgs {
    const int32_t *rows;
    const double *gpart;
    int wg_per_row, n_gslots;
    const int32_t *sym_begin, *sym_gslots, *gslot_slot;
    const double *slot_scale;
    int uniform, n_slots;
    int S;
    float *grad;
};

struct SampArgs {
    const float2 *state;
    int64_t row_stride;
    const int32_t *rows;   // state rows (NULL: the row index)
    const int32_t *brows;  // batch index of each row (NULL: the row index)
    uint64_t *levels;
    int64_t row_level;  // entries per row
    int nlev;           // stored levels 1..nlev; level nlev has at most 64 entries
    int64_t count[kMaxLevels + 1];
    int64_t off[kMaxLevels + 1];
    int64_t n_shots;
    uint64_t seed;
    uint64_t *out;
    int vec16;          // rows start 16-byte aligned (16-byte loads in level 1)
};

// Per-row table offsets of derived rows: out[j][r] = in[j][(x_begin + r) / x_period].
constexpr int kRowGatherArrays = 6;
struct RowGatherArgs {
    const int32_t *in[kRowGatherArrays];
    int32_t *out[kRowGatherArrays];
    int narrays;
    int64_t x_begin;
    int32_t x_period;
    int32_t count;
};

// Expectations estimated from measurement shots (SampledExpectation): each
// non-identity term of an observable measured `reps` times from its exact
// expectation.  Launch row r is a row of term values tv[r][Kt]; its
// observable tables are those of batch row b and its shot counters those of
// row e: plain rows (x_period = 0) have b = e = r; derived rows of a group
// have source group row s = (x_begin + r) / x_period, b = rows[s] and
// e = ebase[s] + (x_begin + r) % x_period.
struct SampledArgs {
    const float *tv;         // [nrows][Kt] term expectations
    int Kt;
    int K;
    int reps;
    uint64_t seed;
    // tables (row stride 0 when every row has the same terms)
    const int32_t *slot_k, *slot_t;  // [.][Kt]: observable and term index of term slot j (t < 0: none)
    int64_t slot_stride;
    const int32_t *obs_begin;        // [.][K + 1]: CSR of each observable's terms
    int64_t obs_stride;
    const int32_t *term_slot;        // term -> its slot j (-1: identity term)
    const double *term_coeff;
    int64_t term_stride;             // terms per table row
    // derived rows
    const int32_t *rows;
    const int64_t *ebase;
    int64_t x_begin;
    int32_t x_period;
    int32_t nrows;
    int64_t w_begin;         // first (row, term slot) pair of a counts launch
    uint32_t *counts;        // [nrows][Kt]
    float *out;              // [nrows][K]
};

// Gradients of the batched shift rules from the expectations of the derived
// rows: per group row s and symbol, the sum over the symbol's move pairs p
// (rows 2p and 2p + 1 of s's expansion, moved + and -) of
// coef_p x scale x sum_k g_k (f_k(+) - f_k(-)), in pair order; scale is the
// row's scale of slot_p (1 when slot_p < 0).
struct ShiftGradArgs {
    const float *f;          // [group rows x period][K], row s x period + j
    int K, S;
    int32_t period;
    const int32_t *rows;     // group row -> batch row
    const float *upstream;   // [B][K]
    const int32_t *sym_begin, *sym_pairs;  // CSR symbol -> pairs
    const int32_t *pair_slot;
    const double *pair_coef;
    double coef_mul;         // every coefficient times this
    const double *slot_scale;
    int uniform, n_slots;
    float *grad;             // [B][S]
};

struct GatherArgs {
    const float2 *state;
    int64_t row_stride;
    const int32_t *rows;   // state rows (NULL: row r is state row r)
    const int32_t *brows;  // batch index of each row (NULL: row r is batch row r)
    int n;
    const uint64_t *bits;
    int64_t M;
    float2 *out;
};

} // namespace tq
