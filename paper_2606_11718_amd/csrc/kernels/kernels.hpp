// Kernel launchers of the CCL library (device side lives in *.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../host/plan.hpp"

namespace ccl {

// Operand addressing of the GEMM kernel, in elements. Logical element
// (m, k) of A with m in partition row pr and k in K-slice kc sits at
//   A + pr * a_part + kc * a_slice + (m - pr*hr) * a_ld + (k - kc*a_kslice)
// (B and C likewise). CCL: a_part = Gc*S, a_slice = S, a_ld = K/Gc.
struct OperandAddr {
  int64_t part;     // stride between partition blocks along the tile grid
  int64_t slice;    // stride between K slices (A, B) / grid columns (C)
  int32_t ld;       // leading dimension inside a block
  int32_t kslice;   // K extent of one block (A, B); unused for C
};

// Pack (row-major -> CCL) or unpack (CCL -> row-major) with ld.
hipError_t launch_copy(const Plan& p, int op, const void* rowmajor, int64_t ld, void* ccl_buf,
                       bool unpack, hipStream_t stream);
// Pack from a stored transpose (cols x rows, leading dimension ld).
hipError_t launch_pack_trans(const Plan& p, int op, const void* src, int64_t ld, void* dst,
                             hipStream_t stream);
// C = alpha A B + beta C with the given operand addressing; remap =
// XCD-aware tile map. C is read only when beta != 0. splits > 1 (remap
// only): split-K into the fp32 workspace ws, then a reduce launch.
// timeline (bf16, unsplit only): kTimelineWords uint64 per wave of every
// workgroup that has a tile, recorded by the kernel (debug launches).
hipError_t launch_gemm(const Plan& p, const void* A, const void* B, void* C,
                       const OperandAddr& a, const OperandAddr& b, const OperandAddr& c,
                       bool remap, float alpha, float beta, int splits, float* ws,
                       hipStream_t stream, uint64_t* timeline = nullptr);
constexpr int kTimelineWords = 8;
// Split-K workspace for callers that cannot allocate device memory: a
// static device array of kScratchBytes in the library (one per GPU, held
// until the process ends). Returns its address on the current device,
// looked up once per device.
constexpr int64_t kScratchBytes = (int64_t)64 << 20;
hipError_t scratch_workspace(float** ws);
// Dispatch probe with the GEMM grid (4 int32 per workgroup).
hipError_t launch_dispatch_probe(const Plan& p, int32_t* out, hipStream_t stream);

}  // namespace ccl
