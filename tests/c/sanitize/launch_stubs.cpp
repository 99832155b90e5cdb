// Recording stand-ins for the kernel launchers of kernels.hpp, linked into the
// sanitizer build of the C-ABI layer instead of the HIP kernels. Each call
// checks what a launch may rely on (pointers set, the plan's GEMM supported,
// split-K with a workspace) and counts itself; nothing is dereferenced.
#include <cstdint>
#include <cstdio>
#include <cstdlib>

#include "kernels/kernels.hpp"

namespace {
long g_launches = 0;

void require(bool ok, const char* what) {
  if (!ok) {
    std::fprintf(stderr, "launch stub: %s\n", what);
    std::abort();
  }
}
}  // namespace

extern "C" long stub_launches(void) { return g_launches; }

namespace ccl {

hipError_t launch_copy(const Plan& p, int op, const void* rowmajor, int64_t ld, void* ccl_buf,
                       bool, hipStream_t) {
  require(rowmajor && ccl_buf && op >= 0 && op < 3 && ld >= p.lay[op].cols, "copy arguments");
  ++g_launches;
  return hipSuccess;
}

hipError_t launch_pack_trans(const Plan& p, int op, const void* src, int64_t ld, void* dst,
                             hipStream_t) {
  require(src && dst && op >= 0 && op < 2 && ld >= p.lay[op].rows, "pack_trans arguments");
  ++g_launches;
  return hipSuccess;
}

hipError_t launch_gemm(const Plan& p, const void* A, const void* B, void* C, const OperandAddr& a,
                       const OperandAddr& b, const OperandAddr&, bool remap, float, float,
                       int splits, float* ws, hipStream_t, uint64_t* timeline) {
  require(A && B && C && p.gemm.supported, "gemm arguments");
  require(!timeline || (splits == 1 && p.ab_type == DT_BF16), "timeline arguments");
  require(a.ld > 0 && b.ld > 0 && a.kslice > 0 && b.kslice > 0, "gemm addressing");
  require(splits >= 1 && (splits == 1 || (ws != nullptr && remap)), "split-K arguments");
  ++g_launches;
  return hipSuccess;
}

hipError_t scratch_workspace(float** ws) {
  *ws = reinterpret_cast<float*>(static_cast<uintptr_t>(1) << 20);   // never dereferenced
  return hipSuccess;
}

hipError_t launch_dispatch_probe(const Plan& p, int32_t* out, hipStream_t) {
  require(out && p.gemm.supported, "dispatch probe arguments");
  ++g_launches;
  return hipSuccess;
}

}  // namespace ccl
