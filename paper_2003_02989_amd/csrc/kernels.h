// kernels.h -- launchers of the libtq kernels.
#pragma once
#include <hip/hip_runtime.h>

#include "kernel_args.h"

namespace tq {


// Opt-in profiler: while `name` is the selected kernel (profile_start), the
// launches made inside a ProfScope are bracketed by a pair of HIP events
// recorded on the launch stream.
struct ProfScope {
    hipEvent_t b = nullptr, e = nullptr;
    hipStream_t s;
    ProfScope(const char *name, hipStream_t st);
    ~ProfScope();
    ProfScope(const ProfScope &) = delete;
    ProfScope &operator=(const ProfScope &) = delete;
};
void profile_start(const char *kernel);
hipError_t profile_read(int64_t *launches, double *total_ms);
// The builder's gate table on the host: the matrix (deriv = 0) or its
// derivative with respect to parameter `which` of opcode `op` at resolved
// parameters eta, as the device builds it (without the global phase it leaves
// out), in `form`; out receives d*d complex entries (re, im); returns d (0 for
// an opcode without that matrix).
int gate_table_host(int op, const double *eta, const double *ex, int form, int deriv, int which, double *out);
size_t pass_lds_bytes(const TileGeom &g, bool product_init, int nmat);
size_t resident_lds_bytes(int n, int nacc, bool adjoint);
hipError_t launch_resident(const ResArgs &a, int nrows, hipStream_t s);
hipError_t launch_build(const BuildArgs &a, int nrows, hipStream_t s);
// derived rows: the source rows' blocks copied, then the listed tasks of each
// row's move rebuilt (max_list: the longest list)
hipError_t launch_build_derived(const BuildArgs &a, int nrows, int max_list, hipStream_t s);
hipError_t launch_build_stage(const StageBuildArgs &a, int nrows, hipStream_t s);
hipError_t launch_pass(const PassArgs &a, int nrows, hipStream_t s);
// Tiles of the Pauli kernel: 2^t amplitudes with t <= kPauliTileMax.
constexpr int kPauliTileMax = 12;
size_t pauli_lds_bytes(const TileGeom &g, int k_count, bool partner);
hipError_t launch_pauli(const PauliArgs &a, int nrows, bool partner, hipStream_t s);
// Workgroups of the diagonal kernel that fit on the device at once (0 if unknown).
int pauli_diag_slots(int amax, int k_count);
// amax: the largest class count of a chunk (<= kDiagClassMax)
hipError_t launch_pauli_diag(const DiagArgs &a, int nrows, int amax, hipStream_t s);
hipError_t launch_pauli_reduce(const PauliReduceArgs &a, int nrows, hipStream_t s);
size_t rev_pass_lds_bytes(const RevArgs &a);
hipError_t launch_rev_pass(const RevArgs &a, int nrows, hipStream_t s);
hipError_t launch_grad_reduce(const GradReduceArgs &a, int nrows, hipStream_t s);
hipError_t launch_sample(const SampArgs &a, int nrows, hipStream_t s);
// The static sampler workspace: kStaticLevelEntries uint64 per device (32 MiB),
// its device address on the current device (looked up on the first call per
// device).
constexpr int64_t kStaticLevelEntries = (int64_t)1 << 22;
hipError_t static_levels(uint64_t **ptr);
hipError_t launch_gather(const GatherArgs &a, int nrows, hipStream_t s);
hipError_t launch_row_mean(const float *in, int64_t groups, int32_t R, int32_t K, float *out, hipStream_t s);
hipError_t launch_row_gather(const RowGatherArgs &a, hipStream_t s);
// shot counts and estimates of the sampled expectation (a.nrows rows)
hipError_t launch_sampled(const SampledArgs &a, hipStream_t s);
hipError_t launch_shift_grad(const ShiftGradArgs &a, int nrows, hipStream_t s);
hipError_t launch_zero_tail(float2 *state, int64_t row_stride, const int32_t *rows, int nrows, int64_t from,
                            int64_t to, hipStream_t s);

} // namespace tq
