// jit.h -- kernels specialised for one circuit structure at run time.
//
// The resident-circuit kernel interprets its stage and op tables: every op
// costs a table read, a dispatch on its kind and register bits, and the
// registers the generic code keeps live.  For a structure that is run many
// times the same computation can be compiled with the tables as constants:
// each stage becomes straight-line code over its register bits, each op a
// call of the register-op template it dispatches to, each matrix read a
// scalar load at a fixed offset of the row's matrix block.  The source is
// generated from the plan, compiled with hipRTC for the current device and
// cached by its text for the life of the process.
#pragma once
#include <hip/hip_runtime.h>

#include <string>

#include "kernel_args.h"
#include "program.h"

namespace tq {

// The specialised resident kernel's source (without the shared device code).
std::string resident_source(const Group &g);

// Launch the specialised resident kernel of group g (compiled on first use
// on the current device).  On a compile failure returns hipErrorInvalidSource
// and sets *log to the compiler's message.
hipError_t launch_resident_spec(const Group &g, const ResArgs &a, int nrows, size_t lds, hipStream_t s,
                                std::string *log);

// Compile the specialised resident kernel of group g ahead of its first
// launch: for the current device when target is NULL (the kernel is then
// cached), else only check that it compiles for the offload target (e.g.
// "gfx950"), which needs no device.
hipError_t prepare_resident_spec(const Group &g, const char *target, std::string *log);

// Specialised kernels compiled so far in this process (all devices).
int spec_kernels_compiled();

} // namespace tq
