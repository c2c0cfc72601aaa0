// jit.cpp -- generation, run-time compilation and launch of the resident
// kernel specialised for one circuit structure.  The generated code calls the
// same register-op templates (device_ops.h) the precompiled kernel dispatches
// to, with the register bits, tile bits and matrix offsets of every op and
// stage written in as constants.
#include "jit.h"

#include "kernels.h"

#include <hip/hiprtc.h>

#include <map>
#include <memory>
#include <mutex>
#include <sstream>
#include <vector>

namespace tq {
namespace {

// tq_internal.h, kernel_args.h and device_ops.h as one text (written by the
// build from the headers, with their local includes removed)
const char kPrelude[] =
#include "jit_prelude.inc"
    ;

std::string N(long v) { return std::to_string(v); }

uint32_t host_sw(uint32_t i) { return i ^ ((i >> 5) & 31u); }

// the item's bit at tile position l (every qubit of a resident circuit is a
// tile bit; a position outside the tile reads as 0, the fixed bits of the
// single tile)
std::string bit(uint8_t l) { return l == kFixed ? std::string("0u") : "((base >> " + N(l) + ") & 1u)"; }
std::string ent(int mat) { return "M[" + N(mat) + "]"; }

// Arguments of the diagonal entries of op on register array `v` with matrix
// offset `mat`: returns the call of rd1/rd2/rscale (or its _dot form).
std::string diag_call(const PassOp &op, int R, int mat, bool dot)
{
    const std::string sfx = dot ? "_dot" : "", args = dot ? "v, f" : "v";
    const std::string Rs = N(R);
    if (op.kind == K_D1) {
        if (op.s0 != kFixed)
            return "rd1" + sfx + "<" + Rs + ", " + N(op.s0) + ">(" + args + ", " + ent(mat) + ", " + ent(mat + 1) + ")";
        return "rscale" + sfx + "<" + Rs + ">(" + args + ", zsel(" + bit(op.l0) + ", " + ent(mat) + ", " +
               ent(mat + 1) + "))";
    }
    const bool r0 = op.s0 != kFixed, r1 = op.s1 != kFixed;
    if (r0 && r1) {
        const int j0 = std::min(op.s0, op.s1), j1 = std::max(op.s0, op.s1);
        const bool q0lo = op.s0 < op.s1;
        const int e[4] = {0, q0lo ? 1 : 2, q0lo ? 2 : 1, 3};
        return "rd2" + sfx + "<" + Rs + ", " + N(j0) + ", " + N(j1) + ">(" + args + ", " + ent(mat + e[0]) + ", " +
               ent(mat + e[1]) + ", " + ent(mat + e[2]) + ", " + ent(mat + e[3]) + ")";
    }
    if (r0) {  // entries (v, 2 + v) with v the bit of q1
        const std::string b = bit(op.l1);
        return "rd1" + sfx + "<" + Rs + ", " + N(op.s0) + ">(" + args + ", zsel(" + b + ", " + ent(mat) + ", " +
               ent(mat + 1) + "), zsel(" + b + ", " + ent(mat + 2) + ", " + ent(mat + 3) + "))";
    }
    if (r1) {  // entries (2v, 2v + 1) with v the bit of q0
        const std::string b = bit(op.l0);
        return "rd1" + sfx + "<" + Rs + ", " + N(op.s1) + ">(" + args + ", zsel(" + b + ", " + ent(mat) + ", " +
               ent(mat + 2) + "), zsel(" + b + ", " + ent(mat + 1) + ", " + ent(mat + 3) + "))";
    }
    const std::string b0 = bit(op.l0), b1 = bit(op.l1);
    return "rscale" + sfx + "<" + Rs + ">(" + args + ", zsel(" + b0 + ", zsel(" + b1 + ", " + ent(mat) + ", " +
           ent(mat + 1) + "), zsel(" + b1 + ", " + ent(mat + 2) + ", " + ent(mat + 3) + ")))";
}

// op applied to register array `v` (matrix at offset mat)
std::string apply(const PassOp &op, int R, int mat, const char *v)
{
    const std::string Rs = N(R), m = "M + " + N(mat), V = v;
    switch (op.kind) {
    case K_M1:
        if (!op.ctrl) return "rm1<" + Rs + ", " + N(op.s0) + ">(" + V + ", " + m + ");";
        if (op.s1 != kFixed) return "rm1c<" + Rs + ", " + N(op.s0) + ", " + N(op.s1) + ">(" + V + ", " + m + ");";
        return "rm1<" + Rs + ", " + N(op.s0) + ">(" + V + ", ctrl_sel(" + m + ", " + bit(op.l1) + " == " +
               N(op.cval) + "u));";
    case K_M2: return "rm2<" + Rs + ", " + N(op.s0) + ", " + N(op.s1) + ">(" + V + ", " + m + ");";
    case K_F2: return "rf2<" + Rs + ", " + N(op.s0) + ", " + N(op.s1) + ">(" + V + ", " + m + ");";
    case K_P2:
        return "rp2<" + Rs + ", " + N(std::min(op.s0, op.s1)) + ", " + N(std::max(op.s0, op.s1)) + ">(" + V + ", " +
               ent(mat) + ", " + ent(mat + 1) + ", " + (op.ptype == 2 ? "-1.0" : "1.0") + ");";
    default: {
        std::string c = diag_call(op, R, mat, false);
        return c.replace(c.find("(v"), 2, "(" + V) + ";";
    }
    }
}

// sum of Re(conj(f) dW v) for the derivative matrix at offset d
std::string dot(const PassOp &op, int R, int d)
{
    const std::string Rs = N(R), m = "M + " + N(d);
    switch (op.kind) {
    case K_M1:
        if (!op.ctrl) return "rm1_dot<" + Rs + ", " + N(op.s0) + ">(v, f, " + m + ")";
        if (op.s1 != kFixed) return "rm1c_dot<" + Rs + ", " + N(op.s0) + ", " + N(op.s1) + ">(v, f, " + m + ")";
        // an item whose control is off sees the identity and a zero derivative
        return "(" + bit(op.l1) + " == " + N(op.cval) + "u ? rm1_dot<" + Rs + ", " + N(op.s0) + ">(v, f, " + m +
               ") : 0.0)";
    case K_M2: return "rm2_dot<" + Rs + ", " + N(op.s0) + ", " + N(op.s1) + ">(v, f, " + m + ")";
    case K_F2: return "rf2_dot<" + Rs + ", " + N(op.s0) + ", " + N(op.s1) + ">(v, f, " + m + ")";
    case K_P2:
        return "rp2_dot<" + Rs + ", " + N(std::min(op.s0, op.s1)) + ", " + N(std::max(op.s0, op.s1)) + ">(v, f, " +
               ent(d) + ", " + ent(d + 1) + ", " + (op.ptype == 2 ? "-1.0" : "1.0") + ")";
    default: return diag_call(op, R, d, true);
    }
}

// item loop header of a stage: base index of the item and the swizzled
// LDS offsets of its 2^R registers
void stage_head(std::ostream &o, const Stage &st, int n, std::vector<uint32_t> &off)
{
    const int R = st.r;
    off.assign(1u << R, 0);
    for (uint32_t k = 0; k < (1u << R); k++) {
        uint32_t x = 0;
        for (int j = 0; j < R; j++)
            if ((k >> j) & 1) x |= 1u << st.bits[j];
        off[k] = host_sw(x);  // sw is linear over xor: sw(base | x) = sw(base) ^ sw(x)
    }
    o << "    for (uint32_t item = tid; item < " << (1u << (n - R)) << "u; item += 256u) {\n";
    o << "        uint32_t base = item;\n";
    for (int j = 0; j < R; j++) o << "        base = ins0(base, " << (int)st.bits[j] << ");\n";
    o << "        const uint32_t sb = sw(base);\n";
}

const std::vector<PassOp> &pass_ops(const Pass &ps) { return ps.ops; }

} // namespace

std::string resident_source(const Group &g)
{
    std::ostringstream o;
    const int n = g.n;
    o << "namespace tq {\n"
         "__device__ __forceinline__ double2 zsel(uint32_t c, double2 a, double2 b) { return c ? b : a; }\n"
         "extern \"C\" __global__ __launch_bounds__(256, 4) void tq_resident_spec(ResArgs a)\n{\n"
         "    extern __shared__ __align__(16) unsigned char smem[];\n"
         "    double *acc = reinterpret_cast<double *>(smem);\n"
         "    float2 *lp = reinterpret_cast<float2 *>(acc + 4 * a.nacc);\n"
         "    float2 *lf = lp + "
      << (1u << n)
      << "u;\n"
         "    const SMat M = smat(a.mats + (int64_t)blockIdx.x * a.mat_stride);\n"
         "    const int tid = threadIdx.x;\n"
         "    resident_begin(a, M, acc, lp, tid, 256);\n";
    std::vector<uint32_t> off;
    for (const Pass &ps : g.fwd)
        for (const Stage &st : ps.stages) {
            const int R = st.r, NR = 1 << R;
            o << "    {\n";
            stage_head(o, st, n, off);
            o << "        double2 v[" << NR << "];\n";
            for (int k = 0; k < NR; k++) o << "        v[" << k << "] = up2(lp[sb ^ " << off[k] << "u]);\n";
            if (st.dense) {
                o << "        rdense<" << R << ">(v, M + " << st.mat << ");\n";
            } else {
                for (int oi = st.op_begin; oi < st.op_end; oi++) {
                    const PassOp &op = pass_ops(ps)[oi - ps.op_offset];
                    o << "        " << apply(op, R, op.mat, "v") << "\n";
                }
            }
            for (int k = 0; k < NR; k++) o << "        lp[sb ^ " << off[k] << "u] = down2(v[" << k << "]);\n";
            o << "    }\n    }\n    __syncthreads();\n";
        }
    o << "    resident_middle(a, acc, lp, lf, blockIdx.x, tid, 256);\n"
         "    if (a.grad) {\n";
    for (const Pass &ps : g.rev)
        for (const Stage &st : ps.stages) {
            const int R = st.r, NR = 1 << R;
            std::vector<std::pair<int, int>> grads;  // (accumulator, gradient slot)
            for (int oi = st.op_begin; oi < st.op_end; oi++) {
                const PassOp &op = pass_ops(ps)[oi - ps.op_offset];
                for (int j = 0; j < op.ngrad; j++) grads.emplace_back((int)grads.size(), op.gslot[j]);
            }
            o << "    {\n";
            if (!grads.empty()) o << "    double g[" << grads.size() << "] = {};\n";
            stage_head(o, st, n, off);
            o << "        double2 v[" << NR << "], f[" << NR << "];\n";
            for (int k = 0; k < NR; k++)
                o << "        v[" << k << "] = up2(lp[sb ^ " << off[k] << "u]); f[" << k << "] = up2(lf[sb ^ "
                  << off[k] << "u]);\n";
            int gk = 0;
            for (int oi = st.op_begin; oi < st.op_end; oi++) {
                const PassOp &op = pass_ops(ps)[oi - ps.op_offset];
                o << "        " << apply(op, R, op.mat, "v") << "\n";
                for (int j = 0; j < op.ngrad; j++) o << "        g[" << gk++ << "] += " << dot(op, R, op.dmat[j]) << ";\n";
                o << "        " << apply(op, R, op.mat, "f") << "\n";
            }
            for (int k = 0; k < NR; k++)
                o << "        lp[sb ^ " << off[k] << "u] = down2(v[" << k << "]); lf[sb ^ " << off[k]
                  << "u] = down2(f[" << k << "]);\n";
            o << "    }\n";
            for (auto &gs : grads)
                o << "    { const double s_ = wave_sum(g[" << gs.first
                  << "]); if ((tid & 63) == 0) acc[(tid >> 6) * a.nacc + a.gacc + " << gs.second << "] += s_; }\n";
            o << "    }\n    __syncthreads();\n";
        }
    o << "    }\n"
         "    resident_end(a, acc, blockIdx.x, tid, 256);\n"
         "}\n"
         "} // namespace tq\n";
    return o.str();
}

namespace {

struct SpecKernel {
    hipModule_t mod = nullptr;
    hipFunction_t fn = nullptr;
};

std::mutex g_mu;
// (device, source) -> compiled kernel; kept until the process ends
std::map<std::pair<int, std::string>, SpecKernel> g_cache;
int g_compiled = 0;

// Compile the kernel source `body` for offload target `target` into a code
// object.
hipError_t compile_code(const std::string &body, const std::string &target, std::vector<char> *code,
                        std::string *log)
{
    const std::string src = std::string(kPrelude) + "\n" + body;
    hiprtcProgram prog;
    if (hiprtcCreateProgram(&prog, src.c_str(), "tq_resident_spec.hip", 0, nullptr, nullptr) != HIPRTC_SUCCESS) {
        *log = "hiprtcCreateProgram failed";
        return hipErrorInvalidSource;
    }
    const std::string arch = "--offload-arch=" + target;
    // the same code generation flags as the precompiled kernels
    const char *opts[] = {arch.c_str(), "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
                          "-packed-fp32-ops"};
    const hiprtcResult r = hiprtcCompileProgram(prog, 7, opts);
    if (r != HIPRTC_SUCCESS) {
        size_t n = 0;
        hiprtcGetProgramLogSize(prog, &n);
        std::string text(n, '\0');
        if (n) hiprtcGetProgramLog(prog, &text[0]);
        *log = "specialised resident kernel: " + std::string(hiprtcGetErrorString(r)) + "\n" + text;
        hiprtcDestroyProgram(&prog);
        return hipErrorInvalidSource;
    }
    size_t size = 0;
    hiprtcGetCodeSize(prog, &size);
    code->resize(size);
    hiprtcGetCode(prog, code->data());
    hiprtcDestroyProgram(&prog);
    return hipSuccess;
}

hipError_t compile(const std::string &body, int dev, SpecKernel *out, std::string *log)
{
    hipDeviceProp_t prop;
    hipError_t e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) return e;
    std::vector<char> code;
    e = compile_code(body, prop.gcnArchName, &code, log);
    if (e != hipSuccess) return e;
    e = hipModuleLoadData(&out->mod, code.data());
    if (e != hipSuccess) return e;
    e = hipModuleGetFunction(&out->fn, out->mod, "tq_resident_spec");
    if (e == hipSuccess) g_compiled++;
    return e;
}

// the compiled kernel of group g on the current device (compiled on first use)
hipError_t get_kernel(const Group &g, SpecKernel *k, std::string *log)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> l(g_mu);
    auto key = std::make_pair(dev, resident_source(g));
    auto it = g_cache.find(key);
    if (it != g_cache.end()) {
        *k = it->second;
        return hipSuccess;
    }
    e = compile(key.second, dev, k, log);
    if (e == hipSuccess) g_cache.emplace(std::move(key), *k);
    return e;
}

} // namespace

hipError_t launch_resident_spec(const Group &g, const ResArgs &a, int nrows, size_t lds, hipStream_t s,
                                std::string *log)
{
    if (nrows <= 0) return hipSuccess;
    SpecKernel k;
    hipError_t e = get_kernel(g, &k, log);
    if (e != hipSuccess) return e;
    ResArgs args = a;
    void *params[] = {&args};
    ProfScope ps("resident", s);
    return hipModuleLaunchKernel(k.fn, nrows, 1, 1, kThreads, 1, 1, (unsigned)lds, s, params, nullptr);
}

hipError_t prepare_resident_spec(const Group &g, const char *target, std::string *log)
{
    if (target) {
        std::vector<char> code;
        return compile_code(resident_source(g), target, &code, log);
    }
    SpecKernel k;
    return get_kernel(g, &k, log);
}

int spec_kernels_compiled()
{
    std::lock_guard<std::mutex> l(g_mu);
    return g_compiled;
}

} // namespace tq
