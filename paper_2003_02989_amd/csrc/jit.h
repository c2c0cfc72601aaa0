// jit.h -- kernels specialised for one circuit structure at run time.
//
// The resident-circuit kernel and the tile passes interpret their stage and
// op tables: every op costs a table read, a dispatch on its kind and register
// bits, and the registers the generic code keeps live.  For a structure that
// is run many times the same computation can be compiled with the tables as
// constants: each stage becomes straight-line code over its register bits,
// each op a call of the register-op template it dispatches to, each matrix
// read a load at a fixed offset (scalar loads from the row's matrix block in
// the resident kernel, LDS reads in the passes).  The source is generated
// from the plan, compiled with hipRTC for the current device and cached by
// its text for the life of the process.
#pragma once
#include <hip/hip_runtime.h>

#include <string>
#include <vector>

#include "kernel_args.h"
#include "program.h"

namespace tq {

// The specialised resident kernel's source (without the shared device code).
std::string resident_source(const Group &g);
// The specialised forward (tq_fwd_<pass>) and reverse (tq_rev_<pass>) tile
// pass kernels of group g, to be placed in namespace tq after the shared
// device code (all passes of a group are compiled as one program).
std::string pass_kernel_source(const Group &g, int pass);
std::string rev_pass_kernel_source(const Group &g, int pass);

// Handles of one structure's specialised kernels on one device.  The caller
// keeps one per structure (and per kind of kernel) so that repeated launches
// neither regenerate the source nor look it up in the process-wide cache;
// it is reset when the current device changes.
struct SpecMemo {
    int dev = -1;
    std::vector<hipFunction_t> fn;  // by kernel slot, null until looked up
    int slots = -1;                 // pauli_spec_slots' answer, -1 until asked
};

// Launch a specialised kernel of group g, compiled on first use on the
// current device: the resident kernel, or forward / reverse pass `pass` (with
// the arguments the precompiled kernel takes).  On a compile failure these
// return hipErrorInvalidSource and set *log to the compiler's message.
// `memo` (one per group and kind: resident, or the group's passes) may be
// NULL.
hipError_t launch_resident_spec(const Group &g, const ResArgs &a, int nrows, size_t lds, hipStream_t s,
                                std::string *log, SpecMemo *memo);
hipError_t launch_pass_spec(const Group &g, int pass, const PassArgs &a, int nrows, hipStream_t s,
                            std::string *log, SpecMemo *memo);
hipError_t launch_rev_pass_spec(const Group &g, int pass, const RevArgs &a, int nrows, hipStream_t s,
                                std::string *log, SpecMemo *memo);

// Kernels tq_pauli_<pass> computing the expectations of one observable set
// of K observables (the same on every row) pass by pass: each pass's tile
// holds the X bits of its terms; partials go to
// partial[row][npass][wg_per_row][k_count].  Up to 16 observables keep
// register accumulators; larger sets per-wave sums in LDS (K doubles per
// wave).
std::string pauli_spec_source(const std::vector<PauliPass> &passes, int K);
hipError_t launch_pauli_spec(const std::string &src, int pass, const PauliSpecArgs &a, int nrows, hipStream_t s,
                             std::string *log, SpecMemo *memo);
// Kernels tq_hphi_<pass> computing phi = g H psi and <psi|H|psi> for one
// observable H (the same on every row) pass by pass, each pass's tile
// holding the X bits of its terms; partials of the expectation go to
// partial[row][npass][wg_per_row].
std::string hphi_spec_source(const std::vector<PauliPass> &passes);
hipError_t launch_hphi_spec(const std::string &src, int pass, const HPhiArgs &a, int nrows, hipStream_t s,
                            std::string *log, SpecMemo *memo);
// Workgroups of a specialised Pauli pass that fit on the device at once (0 if unknown).
int pauli_spec_slots(const std::string &src, const TileGeom &g, int K, std::string *log, SpecMemo *memo);

// Compile the specialised kernels of group g (the resident kernel, or the
// forward and reverse pass kernels) ahead of their first launch: for the current device when
// target is NULL (the module is then cached), else only check that they
// compile for the offload target (e.g. "gfx950"), which needs no device.
hipError_t prepare_spec(const Group &g, bool resident, const char *target, std::string *log);

// Specialised kernel programs loaded so far in this process (all devices),
// and how many of their code objects came from the on-disk code cache.
int spec_kernels_compiled();
int spec_disk_cache_hits();

} // namespace tq
