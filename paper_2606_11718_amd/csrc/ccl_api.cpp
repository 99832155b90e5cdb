// C ABI of the CCL library (declarations and contracts: include/ccl.h).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <mutex>
#include <exception>
#include <new>
#include <string>

#include "../../include/ccl.h"
#include "host/l2sim.hpp"
#include "host/plan.hpp"
#include "kernels/kernels.hpp"

struct ccl_plan_s {
  ccl::Plan plan;
};

namespace {

thread_local std::string g_last_error;

ccl_status fail(ccl_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

ccl_status ok() {
  g_last_error.clear();
  return CCL_OK;
}

ccl_status from(ccl::Status s, const std::string& msg) {
  return s == ccl::Status::OK ? ok() : fail(static_cast<ccl_status>(s), msg);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// gfx950 check, once per device.
constexpr int kMaxDevices = 64;
std::once_flag g_dev_once[kMaxDevices];
bool g_dev_ok[kMaxDevices];

ccl_status check_device() {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(CCL_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(CCL_ERR_UNSUPPORTED, "device index out of range");
  std::call_once(g_dev_once[dev], [dev] {
    hipDeviceProp_t prop;
    g_dev_ok[dev] = hipGetDeviceProperties(&prop, dev) == hipSuccess &&
                    std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
  });
  if (!g_dev_ok[dev]) return fail(CCL_ERR_UNSUPPORTED, "the GPU kernels are built for gfx950 only");
  return CCL_OK;
}

ccl_status hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(CCL_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
  return ok();
}

bool valid_op(ccl_operand op) { return op == CCL_A || op == CCL_B || op == CCL_C; }

// CCL addressing of the GEMM operands (in elements of each operand's type).
void ccl_addressing(const ccl::Plan& p, ccl::OperandAddr* a, ccl::OperandAddr* b,
                    ccl::OperandAddr* c) {
  const int64_t sa = p.lay[ccl::OP_A].strip_stride_bytes / p.lay[ccl::OP_A].elem_bytes;
  const int64_t sb = p.lay[ccl::OP_B].strip_stride_bytes / p.lay[ccl::OP_B].elem_bytes;
  const int64_t sc = p.lay[ccl::OP_C].strip_stride_bytes / p.lay[ccl::OP_C].elem_bytes;
  // A block (pr, kc) = pr*Gc + kc; B block (kr, pc) = kr*Gc + pc; C block (pr, pc).
  *a = {p.Gc * sa, sa, (int32_t)(p.K / p.Gc), (int32_t)(p.K / p.Gc)};
  *b = {sb, p.Gc * sb, (int32_t)(p.N / p.Gc), (int32_t)(p.K / p.Gr)};
  *c = {p.Gc * sc, sc, (int32_t)(p.N / p.Gc), 0};
}

// Row-major addressing of the same operands (Eq. 2): A (M x K), B (K x N),
// C (M x N), leading dimensions K, N, N.
void rowmajor_addressing(const ccl::Plan& p, ccl::OperandAddr* a, ccl::OperandAddr* b,
                         ccl::OperandAddr* c) {
  const int64_t hr = p.M / p.Gr;
  *a = {hr * p.K, p.K / p.Gc, (int32_t)p.K, (int32_t)(p.K / p.Gc)};
  *b = {p.N / p.Gc, (p.K / p.Gr) * p.N, (int32_t)p.N, (int32_t)(p.K / p.Gr)};
  *c = {hr * p.N, p.N / p.Gc, (int32_t)p.N, 0};
}

// Whether every element the GEMM kernel can touch through this addressing
// lies inside buffers of a_bytes, b_bytes and c_bytes (the kernel's own
// formulas: A at pr*part + kslice_index*slice + row*ld + k, B at
// pc*part + kslice_index*slice + k*ld + n, C at pr*part + pc*slice +
// row*ld + n).
bool addressing_in_bounds(const ccl::Plan& p, const ccl::OperandAddr& a, const ccl::OperandAddr& b,
                          const ccl::OperandAddr& c, int64_t a_bytes, int64_t b_bytes,
                          int64_t c_bytes) {
  const int64_t hr = p.M / p.Gr, wc = p.N / p.Gc;
  const int64_t a_end = (p.Gr - 1) * a.part + (p.K / a.kslice - 1) * a.slice + (hr - 1) * a.ld + a.kslice;
  const int64_t b_end = (p.Gc - 1) * b.part + (p.K / b.kslice - 1) * b.slice + (b.kslice - 1) * b.ld + wc;
  const int64_t c_end = (p.Gr - 1) * c.part + (p.Gc - 1) * c.slice + (hr - 1) * c.ld + wc;
  return a_end * p.lay[ccl::OP_A].elem_bytes <= a_bytes &&
         b_end * p.lay[ccl::OP_B].elem_bytes <= b_bytes &&
         c_end * p.lay[ccl::OP_C].elem_bytes <= c_bytes;
}

// The kernels address a tile's K steps with 32-bit byte offsets and 32-bit
// buffer sizes from the tile corner. The widest spans any kernel builds:
// A, 255 rows plus four bf16 K steps (256 bytes); B, 127 rows (four bf16
// steps of the rounds path, or one 128-wide fp8 step) plus a 256-column
// row. Both must stay below 2^31 (less a page of margin), whichever kernel
// the plan selects.
bool offsets_fit(const ccl::Plan& p, const ccl::OperandAddr& a, const ccl::OperandAddr& b) {
  const int64_t lim = ((int64_t)1 << 31) - 4096;
  const int64_t e = p.lay[ccl::OP_A].elem_bytes;
  return 255 * (int64_t)a.ld * e + 256 < lim && 127 * (int64_t)b.ld * e + 256 * e < lim;
}

}  // namespace

extern "C" {

ccl_status ccl_plan_typed(int64_t M, int64_t N, int64_t K, int chiplets, int grid_rows,
                          int64_t page_bytes, ccl_dtype ab_type, ccl_dtype c_type, ccl_plan_t* out) {
  if (!out) return fail(CCL_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  ccl::Plan p;
  std::string err;
  ccl::Status s = ccl::make_plan(M, N, K, chiplets, grid_rows, page_bytes,
                                 static_cast<ccl::DType>(ab_type), static_cast<ccl::DType>(c_type),
                                 &p, &err);
  if (s != ccl::Status::OK) return from(s, err);
  ccl_plan_s* h = new (std::nothrow) ccl_plan_s;
  if (!h) return fail(CCL_ERR_INVALID_ARG, "out of host memory");
  h->plan = p;
  *out = h;
  return ok();
}

ccl_status ccl_plan(int64_t M, int64_t N, int64_t K, int chiplets, int grid_rows,
                    int64_t page_bytes, ccl_plan_t* out) {
  return ccl_plan_typed(M, N, K, chiplets, grid_rows, page_bytes, CCL_DT_BF16, CCL_DT_BF16, out);
}

ccl_status ccl_plan_destroy(ccl_plan_t plan) {
  delete plan;
  return ok();
}

ccl_status ccl_plan_grid(ccl_plan_t plan, int* grid_rows, int* grid_cols) {
  if (!plan || !grid_rows || !grid_cols) return fail(CCL_ERR_INVALID_ARG, "NULL argument");
  *grid_rows = plan->plan.Gr;
  *grid_cols = plan->plan.Gc;
  return ok();
}

ccl_status ccl_plan_layout(ccl_plan_t plan, ccl_operand op, ccl_layout* out) {
  if (!plan || !out) return fail(CCL_ERR_INVALID_ARG, "NULL argument");
  if (!valid_op(op)) return fail(CCL_ERR_INVALID_ARG, "operand must be CCL_A, CCL_B or CCL_C");
  const ccl::Layout& l = plan->plan.lay[op];
  out->rows = l.rows;
  out->cols = l.cols;
  out->grid_r = l.grid_r;
  out->grid_c = l.grid_c;
  out->block_rows = l.block_rows;
  out->block_cols = l.block_cols;
  out->strip_bytes = l.strip_bytes;
  out->strip_stride_bytes = l.strip_stride_bytes;
  out->total_bytes = l.total_bytes;
  out->elem_bytes = l.elem_bytes;
  return ok();
}

ccl_status ccl_pack(ccl_plan_t plan, ccl_operand op, const void* src, int64_t ld, int src_trans,
                    void* dst_ccl, void* stream) {
  if (!plan || !src || !dst_ccl) return fail(CCL_ERR_INVALID_ARG, "NULL argument");
  if (!valid_op(op)) return fail(CCL_ERR_INVALID_ARG, "operand must be CCL_A, CCL_B or CCL_C");
  if (src_trans != 0 && src_trans != 1) return fail(CCL_ERR_INVALID_ARG, "src_trans must be 0 or 1");
  if (src_trans && op == CCL_C) return fail(CCL_ERR_INVALID_ARG, "C has no stored-transpose form");
  const ccl::Layout& l = plan->plan.lay[op];
  if (ld < (src_trans ? l.rows : l.cols)) return fail(CCL_ERR_INVALID_ARG, "ld is smaller than the stored row");
  if (l.block_rows * l.block_cols >= ((int64_t)1 << 31))
    return fail(CCL_ERR_UNSUPPORTED, "a CCL strip of 2^31 elements or more is not supported");
  if (ccl_status s = check_device()) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (src_trans) return hip_status(ccl::launch_pack_trans(plan->plan, op, src, ld, dst_ccl, st), "pack_trans launch");
  return hip_status(ccl::launch_copy(plan->plan, op, src, ld, dst_ccl, false, st), "pack launch");
}

ccl_status ccl_unpack(ccl_plan_t plan, ccl_operand op, const void* src_ccl, void* dst, int64_t ld,
                      void* stream) {
  if (!plan || !src_ccl || !dst) return fail(CCL_ERR_INVALID_ARG, "NULL argument");
  if (!valid_op(op)) return fail(CCL_ERR_INVALID_ARG, "operand must be CCL_A, CCL_B or CCL_C");
  const ccl::Layout& l = plan->plan.lay[op];
  if (ld < l.cols) return fail(CCL_ERR_INVALID_ARG, "ld is smaller than the operand's columns");
  if (l.block_rows * l.block_cols >= ((int64_t)1 << 31))
    return fail(CCL_ERR_UNSUPPORTED, "a CCL strip of 2^31 elements or more is not supported");
  if (ccl_status s = check_device()) return s;
  return hip_status(ccl::launch_copy(plan->plan, op, dst, ld, const_cast<void*>(src_ccl), true,
                                     static_cast<hipStream_t>(stream)),
                    "unpack launch");
}

ccl_status ccl_gemm_scaled(ccl_plan_t plan, float alpha, const void* A_ccl, const void* B_ccl,
                           float beta, void* C_ccl, void* stream) {
  if (!plan || !A_ccl || !B_ccl || !C_ccl) return fail(CCL_ERR_INVALID_ARG, "NULL argument");
  if (!aligned16(A_ccl) || !aligned16(B_ccl) || !aligned16(C_ccl))
    return fail(CCL_ERR_MISALIGNED_POINTER, "A, B and C must be 16-byte aligned");
  const ccl::Plan& p = plan->plan;
  if (!p.gemm.supported) return fail(CCL_ERR_UNSUPPORTED, p.gemm.why_unsupported);
  ccl::OperandAddr a, b, c;
  ccl_addressing(p, &a, &b, &c);
  if (!offsets_fit(p, a, b)) return fail(CCL_ERR_UNSUPPORTED, "CCL blocks too wide for 32-bit in-tile offsets");
  if (!addressing_in_bounds(p, a, b, c, p.lay[ccl::OP_A].total_bytes, p.lay[ccl::OP_B].total_bytes,
                            p.lay[ccl::OP_C].total_bytes))
    return fail(CCL_ERR_UNSUPPORTED, "internal error: GEMM addressing exceeds the CCL buffers");
  if (ccl_status s = check_device()) return s;
  return hip_status(ccl::launch_gemm(p, A_ccl, B_ccl, C_ccl, a, b, c, true, alpha, beta, 1,
                                     nullptr, static_cast<hipStream_t>(stream)),
                    "gemm launch");
}

// The split-K launch has about splits times the workgroups of the plain
// GEMM, its reduce launch tile_m * tile_n / 1024 times as many.
static ccl_status check_split_grid(const ccl::Plan& p, int splits) {
  if (ccl::splitk_workgroups(p, splits) > 0x7fffffff ||
      ccl::splitk_reduce_workgroups(p) > 0x7fffffff)
    return fail(CCL_ERR_UNSUPPORTED, "split-K grid exceeds the launch limit");
  return ok();
}

ccl_status ccl_gemm_splitk_workspace(ccl_plan_t plan, int* splits, int64_t* workspace_bytes) {
  if (!plan || !splits || !workspace_bytes) return fail(CCL_ERR_INVALID_ARG, "NULL argument");
  const ccl::Plan& p = plan->plan;
  if (!p.gemm.supported) return fail(CCL_ERR_UNSUPPORTED, p.gemm.why_unsupported);
  int s = *splits == 0 ? ccl::recommended_splits(p) : *splits;
  if (s < 1 || s > ccl::kMaxSplits)
    return fail(CCL_ERR_INVALID_ARG, "splits must be 0 (choose) or in 1..16");
  if (ccl_status st = check_split_grid(p, s)) return st;
  *splits = ccl::effective_splits(p, s);
  *workspace_bytes = ccl::splitk_workspace_bytes(p, s);
  return ok();
}

ccl_status ccl_gemm_splitk(ccl_plan_t plan, float alpha, const void* A_ccl, const void* B_ccl,
                           float beta, void* C_ccl, int splits, void* workspace,
                           int64_t workspace_bytes, void* stream) {
  if (!plan || !A_ccl || !B_ccl || !C_ccl) return fail(CCL_ERR_INVALID_ARG, "NULL argument");
  const ccl::Plan& p = plan->plan;
  if (!p.gemm.supported) return fail(CCL_ERR_UNSUPPORTED, p.gemm.why_unsupported);
  if (splits < 1 || splits > ccl::kMaxSplits)
    return fail(CCL_ERR_INVALID_ARG, "splits must be in 1..16");
  if (ccl::effective_splits(p, splits) == 1)
    return ccl_gemm_scaled(plan, alpha, A_ccl, B_ccl, beta, C_ccl, stream);
  if (ccl_status st = check_split_grid(p, splits)) return st;
  if (!workspace) return fail(CCL_ERR_INVALID_ARG, "NULL workspace");
  if (workspace_bytes < ccl::splitk_workspace_bytes(p, splits))
    return fail(CCL_ERR_INVALID_ARG, "workspace smaller than ccl_gemm_splitk_workspace reports");
  if (!aligned16(A_ccl) || !aligned16(B_ccl) || !aligned16(C_ccl) || !aligned16(workspace))
    return fail(CCL_ERR_MISALIGNED_POINTER, "A, B, C and the workspace must be 16-byte aligned");
  ccl::OperandAddr a, b, c;
  ccl_addressing(p, &a, &b, &c);
  if (!offsets_fit(p, a, b)) return fail(CCL_ERR_UNSUPPORTED, "CCL blocks too wide for 32-bit in-tile offsets");
  if (!addressing_in_bounds(p, a, b, c, p.lay[ccl::OP_A].total_bytes, p.lay[ccl::OP_B].total_bytes,
                            p.lay[ccl::OP_C].total_bytes))
    return fail(CCL_ERR_UNSUPPORTED, "internal error: GEMM addressing exceeds the CCL buffers");
  if (ccl_status s = check_device()) return s;
  return hip_status(ccl::launch_gemm(p, A_ccl, B_ccl, C_ccl, a, b, c, true, alpha, beta, splits,
                                     static_cast<float*>(workspace), static_cast<hipStream_t>(stream)),
                    "split-K gemm launch");
}

ccl_status ccl_gemm_splitk_noalloc(ccl_plan_t plan, float alpha, const void* A_ccl,
                                   const void* B_ccl, float beta, void* C_ccl, int splits,
                                   void* stream) {
  if (!plan || !A_ccl || !B_ccl || !C_ccl) return fail(CCL_ERR_INVALID_ARG, "NULL argument");
  const ccl::Plan& p = plan->plan;
  if (!p.gemm.supported) return fail(CCL_ERR_UNSUPPORTED, p.gemm.why_unsupported);
  if (splits < 1 || splits > ccl::kMaxSplits)
    return fail(CCL_ERR_INVALID_ARG, "splits must be in 1..16");
  if (ccl::effective_splits(p, splits) == 1)
    return ccl_gemm_scaled(plan, alpha, A_ccl, B_ccl, beta, C_ccl, stream);
  if (ccl_status st = check_split_grid(p, splits)) return st;
  const int64_t need = ccl::splitk_workspace_bytes(p, splits);
  if (need > ccl::kScratchBytes)
    return fail(CCL_ERR_INVALID_ARG,
                "split-K workspace of " + std::to_string(need) +
                    " bytes exceeds the library's static scratch of " +
                    std::to_string(ccl::kScratchBytes) +
                    " bytes; use fewer splits or ccl_gemm_splitk with a caller workspace");
  if (!aligned16(A_ccl) || !aligned16(B_ccl) || !aligned16(C_ccl))
    return fail(CCL_ERR_MISALIGNED_POINTER, "A, B and C must be 16-byte aligned");
  if (ccl_status s = check_device()) return s;
  float* ws = nullptr;
  if (ccl_status s = hip_status(ccl::scratch_workspace(&ws), "static scratch lookup")) return s;
  return ccl_gemm_splitk(plan, alpha, A_ccl, B_ccl, beta, C_ccl, splits, ws, ccl::kScratchBytes,
                         stream);
}

ccl_status ccl_gemm(ccl_plan_t plan, const void* A_ccl, const void* B_ccl, void* C_ccl,
                    void* stream) {
  return ccl_gemm_scaled(plan, 1.f, A_ccl, B_ccl, 0.f, C_ccl, stream);
}

ccl_status ccl_gemm_rowmajor(ccl_plan_t plan, const void* A, const void* B, void* C, int remap,
                             void* stream) {
  if (!plan || !A || !B || !C) return fail(CCL_ERR_INVALID_ARG, "NULL argument");
  if (remap != 0 && remap != 1) return fail(CCL_ERR_INVALID_ARG, "remap must be 0 or 1");
  if (!aligned16(A) || !aligned16(B) || !aligned16(C))
    return fail(CCL_ERR_MISALIGNED_POINTER, "A, B and C must be 16-byte aligned");
  const ccl::Plan& p = plan->plan;
  if (!p.gemm.supported) return fail(CCL_ERR_UNSUPPORTED, p.gemm.why_unsupported);
  ccl::OperandAddr a, b, c;
  rowmajor_addressing(p, &a, &b, &c);
  if (!offsets_fit(p, a, b)) return fail(CCL_ERR_UNSUPPORTED, "rows too long for 32-bit in-tile offsets");
  if (!addressing_in_bounds(p, a, b, c, p.M * p.K * p.lay[ccl::OP_A].elem_bytes,
                            p.K * p.N * p.lay[ccl::OP_B].elem_bytes,
                            p.M * p.N * p.lay[ccl::OP_C].elem_bytes))
    return fail(CCL_ERR_UNSUPPORTED, "internal error: GEMM addressing exceeds the operands");
  if (ccl_status s = check_device()) return s;
  return hip_status(ccl::launch_gemm(p, A, B, C, a, b, c, remap == 1, 1.f, 0.f, 1, nullptr,
                                     static_cast<hipStream_t>(stream)),
                    "gemm launch");
}

ccl_status ccl_remote_bytes(ccl_plan_t plan, ccl_placement placement, int flags,
                            ccl_traffic* out) {
  if (!plan || !out) return fail(CCL_ERR_INVALID_ARG, "NULL argument");
  if (placement != CCL_PLACE_RR && placement != CCL_PLACE_COARSE && placement != CCL_PLACE_CCL)
    return fail(CCL_ERR_INVALID_ARG, "unknown placement");
  if (flags < 0 || flags > 7) return fail(CCL_ERR_INVALID_ARG, "flags must be in 0..7");
  ccl::Traffic t = ccl::remote_bytes(plan->plan, static_cast<ccl::Placement>(placement), flags);
  std::memset(out, 0, sizeof(*out));
  for (int i = 0; i < 3; ++i) {
    out->accessed[i] = t.accessed[i];
    out->remote[i] = t.remote[i];
    out->footprint[i] = t.footprint[i];
  }
  out->floor_bytes = t.floor_bytes;
  for (int i = 0; i < t.chiplets; ++i) out->remote_per_chiplet[i] = t.remote_per_chiplet[i];
  out->chiplets = t.chiplets;
  return ok();
}

ccl_status ccl_remote_bytes_l2(ccl_plan_t plan, ccl_placement placement, int flags,
                               const ccl_l2_config* config, ccl_l2_traffic* out) {
  if (!plan || !config || !out) return fail(CCL_ERR_INVALID_ARG, "NULL argument");
  if (placement != CCL_PLACE_RR && placement != CCL_PLACE_COARSE && placement != CCL_PLACE_CCL)
    return fail(CCL_ERR_INVALID_ARG, "unknown placement");
  if (flags < 0 || flags > 7) return fail(CCL_ERR_INVALID_ARG, "flags must be in 0..7");
  ccl::L2Config c;
  c.l2_bytes = config->l2_bytes;
  c.ways = config->ways;
  c.line = config->line_bytes;
  c.slots = config->slots;
  c.k_step = config->k_step;
  c.traversal = config->traversal;
  c.group_rows = config->group_rows;
  c.threads = config->threads;
  std::string why = ccl::check_l2_config(c);
  if (why.empty() && c.line > plan->plan.page) why = "line_bytes must not exceed the page size";
  if (!why.empty()) return fail(CCL_ERR_INVALID_ARG, why);
  ccl::L2Traffic t;
  try {
    t = ccl::remote_bytes_l2(plan->plan, static_cast<ccl::Placement>(placement), flags, c);
  } catch (const std::exception& e) {
    return fail(CCL_ERR_INVALID_ARG, std::string("simulation failed: ") + e.what());
  }
  std::memset(out, 0, sizeof(*out));
  for (int i = 0; i < 2; ++i) {
    out->accesses[i] = t.accesses[i];
    out->misses[i] = t.misses[i];
  }
  for (int i = 0; i < 3; ++i) out->remote[i] = t.remote[i];
  for (int i = 0; i < t.chiplets; ++i) out->remote_per_chiplet[i] = t.remote_per_chiplet[i];
  out->chiplets = t.chiplets;
  return ok();
}

const char* ccl_status_string(ccl_status status) {
  switch (status) {
    case CCL_OK: return "CCL_OK";
    case CCL_ERR_INVALID_ARG: return "CCL_ERR_INVALID_ARG";
    case CCL_ERR_UNALIGNED_PARTITION: return "CCL_ERR_UNALIGNED_PARTITION";
    case CCL_ERR_UNSUPPORTED: return "CCL_ERR_UNSUPPORTED";
    case CCL_ERR_MISALIGNED_POINTER: return "CCL_ERR_MISALIGNED_POINTER";
    case CCL_ERR_HIP: return "CCL_ERR_HIP";
  }
  return "CCL_ERR_UNKNOWN";
}

const char* ccl_last_error(void) { return g_last_error.c_str(); }

ccl_status ccl_debug_tile_of_wg(ccl_plan_t plan, int64_t wg, int* xcd, int64_t* tile_m,
                                int64_t* tile_n) {
  if (!plan || !xcd || !tile_m || !tile_n) return fail(CCL_ERR_INVALID_ARG, "NULL argument");
  if (!plan->plan.gemm.supported) return fail(CCL_ERR_UNSUPPORTED, plan->plan.gemm.why_unsupported);
  ccl::tile_of_wg(plan->plan, wg, xcd, tile_m, tile_n);
  return ok();
}

ccl_status ccl_debug_gemm_config(ccl_plan_t plan, int* tile_rows, int* tile_cols,
                                 int64_t* workgroups) {
  if (!plan || !tile_rows || !tile_cols || !workgroups) return fail(CCL_ERR_INVALID_ARG, "NULL argument");
  if (!plan->plan.gemm.supported) return fail(CCL_ERR_UNSUPPORTED, plan->plan.gemm.why_unsupported);
  *tile_rows = plan->plan.gemm.tile_m;
  *tile_cols = plan->plan.gemm.tile_n;
  *workgroups = plan->plan.gemm.workgroups;
  return ok();
}

ccl_status ccl_debug_gemm_timeline(ccl_plan_t plan, const void* A_ccl, const void* B_ccl,
                                   void* C_ccl, uint64_t* timeline, int64_t timeline_bytes,
                                   void* stream) {
  if (!plan || !A_ccl || !B_ccl || !C_ccl || !timeline)
    return fail(CCL_ERR_INVALID_ARG, "NULL argument");
  const ccl::Plan& p = plan->plan;
  if (!p.gemm.supported) return fail(CCL_ERR_UNSUPPORTED, p.gemm.why_unsupported);
  if (p.ab_type != ccl::DT_BF16)
    return fail(CCL_ERR_UNSUPPORTED, "the timeline is recorded by the bf16 GEMM kernel only");
  const int64_t need = p.gemm.workgroups * p.gemm.waves * ccl::kTimelineWords * 8;
  if (timeline_bytes < need)
    return fail(CCL_ERR_INVALID_ARG, "timeline smaller than workgroups * waves * 64 bytes (" +
                                         std::to_string(need) + ")");
  if (!aligned16(A_ccl) || !aligned16(B_ccl) || !aligned16(C_ccl) || !aligned16(timeline))
    return fail(CCL_ERR_MISALIGNED_POINTER, "A, B, C and the timeline must be 16-byte aligned");
  ccl::OperandAddr a, b, c;
  ccl_addressing(p, &a, &b, &c);
  if (!offsets_fit(p, a, b)) return fail(CCL_ERR_UNSUPPORTED, "CCL blocks too wide for 32-bit in-tile offsets");
  if (!addressing_in_bounds(p, a, b, c, p.lay[ccl::OP_A].total_bytes, p.lay[ccl::OP_B].total_bytes,
                            p.lay[ccl::OP_C].total_bytes))
    return fail(CCL_ERR_UNSUPPORTED, "internal error: GEMM addressing exceeds the CCL buffers");
  if (ccl_status s = check_device()) return s;
  return hip_status(ccl::launch_gemm(p, A_ccl, B_ccl, C_ccl, a, b, c, true, 1.f, 0.f, 1, nullptr,
                                     static_cast<hipStream_t>(stream), timeline),
                    "gemm timeline launch");
}

ccl_status ccl_debug_dispatch(ccl_plan_t plan, int32_t* out, void* stream) {
  if (!plan || !out) return fail(CCL_ERR_INVALID_ARG, "NULL argument");
  if (!plan->plan.gemm.supported) return fail(CCL_ERR_UNSUPPORTED, plan->plan.gemm.why_unsupported);
  if (ccl_status s = check_device()) return s;
  return hip_status(ccl::launch_dispatch_probe(plan->plan, out, static_cast<hipStream_t>(stream)),
                    "dispatch probe launch");
}

}  // extern "C"
