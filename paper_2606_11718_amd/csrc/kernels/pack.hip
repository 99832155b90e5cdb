// Pack / unpack between row-major (or stored-transpose) operands and the
// Chiplet-Contiguous Layout (Sec. III-B, Eq. 3 in block form); elements of
// 1, 2 or 4 bytes (fp8, bf16, fp32) are moved as bits:
//   block b = (r / hr) * Gc + c / wc
//   byte offset = b * S + ((r % hr) * wc + c % wc) * e     (S = padded strip)
//
// The work is enumerated in CCL order: block b, then its q-th element (or
// 16-byte chunk) in strip order, so every thread's CCL access is the next
// contiguous piece of a strip and its row-major access is a contiguous run
// of one row slice. Division by the run length uses a host-computed
// multiplier. These kernels move bytes only; they are bound by HBM.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "kernels.hpp"

namespace ccl {

namespace {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));   // one 16-byte chunk

constexpr int64_t kInfinityCacheBytes = 256ll << 20;          // MI355X MALL
// Workgroups of copy_stream_kernel's resident grid: 8 of 256 threads per CU
// on 256 CUs (2048 measured best of 1024, 2048, 3072 and 4096).
constexpr unsigned kResidentWgs = 2048;

// q / d for q < 2^31, d < 2^31: multiply by ceil(2^s / d), s = 31 + ceil(log2 d).
struct DivMagic {
  uint64_t mul;
  uint32_t shift;
  uint32_t d;
};

DivMagic make_div(uint32_t d) {
  uint32_t l = 0;
  while ((1ull << l) < d) ++l;
  DivMagic m;
  m.shift = 31 + l;
  m.mul = (((uint64_t)1 << m.shift) + d - 1) / d;
  m.d = d;
  return m;
}

__device__ __forceinline__ uint32_t fdiv(uint32_t q, const DivMagic& m) {
  return (uint32_t)(((uint64_t)q * m.mul) >> m.shift);
}

struct PackArgs {
  const char* rm;          // row-major side
  char* rm_out;            // row-major side when written (unpack)
  const char* ccl;         // CCL side (read by unpack)
  char* ccl_out;           // CCL side (written by pack)
  int64_t ld_bytes;        // row-major leading dimension
  int64_t strip;           // padded strip stride, bytes
  int64_t hr;              // block rows
  int64_t row_bytes;       // bytes of one block row (wc * e)
  int32_t grid_c;
  uint32_t units_per_block;  // hr * row_bytes / sizeof(U)
  DivMagic units_per_row;    // row_bytes / sizeof(U)
};

// Load / store one unit; NT = non-temporal (streaming) access.
template <bool NT, typename T>
__device__ __forceinline__ T ld(const T* p) {
  if constexpr (NT) return __builtin_nontemporal_load(p);
  else return *p;
}
template <bool NT, typename T>
__device__ __forceinline__ void st(T* p, T v) {
  if constexpr (NT) __builtin_nontemporal_store(v, p);
  else *p = v;
}

// U = unit moved per access: one 16-byte vector, or one element (1, 2 or 4
// bytes) when rows are not 16-byte multiples. UNPACK = false: row-major ->
// CCL; true: CCL -> row-major. NTL / NTS: streaming (non-temporal) loads /
// stores, used for tensors larger than the 256 MiB Infinity Cache
// (measured: +10 % on a 470 MB copy, -15 % on a 134 MB one that the cache
// holds). Below that size, plain stores let the packed operand land in the
// Infinity Cache: streaming stores made the 134 MB activation pack 12 %
// slower between the FFN GEMMs.
template <typename U, bool UNPACK, bool NTL, bool NTS>
__global__ void __launch_bounds__(256) copy_kernel(PackArgs a) {
  const int32_t b = blockIdx.y;                      // strip / chiplet
  const int64_t pr = b / a.grid_c, pc = b % a.grid_c;
  const int64_t rm_base = pr * a.hr * a.ld_bytes + pc * a.row_bytes;
  const char* src_rm = a.rm + rm_base;
  char* dst_rm = a.rm_out + rm_base;
  const int64_t strip_base = (int64_t)b * a.strip;
  constexpr int UNROLL = 4;
  constexpr int64_t US = sizeof(U);
  const uint32_t stride = gridDim.x * 256u;
  for (uint32_t base = blockIdx.x * 256u * UNROLL; base < a.units_per_block; base += stride * UNROLL) {
    U v[UNROLL];
    int64_t rm_off[UNROLL];
    bool ok[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const uint32_t q = base + threadIdx.x + u * 256u;
      ok[u] = q < a.units_per_block;
      const uint32_t row = fdiv(q, a.units_per_row);
      const uint32_t col = q - row * a.units_per_row.d;
      rm_off[u] = (int64_t)row * a.ld_bytes + (int64_t)col * US;
      if (ok[u]) {
        if (UNPACK)
          v[u] = ld<NTL>(reinterpret_cast<const U*>(a.ccl + strip_base + (int64_t)q * US));
        else
          v[u] = ld<NTL>(reinterpret_cast<const U*>(src_rm + rm_off[u]));
      }
    }
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const uint32_t q = base + threadIdx.x + u * 256u;
      if (ok[u]) {
        if (UNPACK)
          st<NTS>(reinterpret_cast<U*>(dst_rm + rm_off[u]), v[u]);
        else
          st<NTS>(reinterpret_cast<U*>(a.ccl_out + strip_base + (int64_t)q * US), v[u]);
      }
    }
  }
}

// 16-byte units of tensors below the Infinity Cache size: a resident grid
// (about 8 workgroups per CU) walks each strip with a stride of the whole
// grid, and issues the loads of its next round before the stores of the
// current one, so every workgroup keeps a round of loads in flight instead
// of one load-then-store pass per workgroup. Loads stream (the source is
// not read again by the path); stores are plain, so the packed operand can
// stay in the Infinity Cache for the GEMM that reads it next. Measured on
// the 134 MB pack of X from HBM: 5.39-5.41 TB/s against 5.05-5.14 for
// copy_kernel; inside the FFN step 46 us against 54 us.
template <bool UNPACK>
__global__ void __launch_bounds__(256) copy_stream_kernel(PackArgs a) {
  const int32_t b = blockIdx.y;                      // strip / chiplet
  const int64_t pr = b / a.grid_c, pc = b % a.grid_c;
  const int64_t rm_base = pr * a.hr * a.ld_bytes + pc * a.row_bytes;
  const char* src_rm = a.rm + rm_base;
  char* dst_rm = a.rm_out + rm_base;
  const int64_t strip_base = (int64_t)b * a.strip;
  constexpr int UNROLL = 4;
  constexpr uint32_t kRound = 256u * UNROLL;         // units per workgroup round
  const uint32_t stride = gridDim.x * kRound;
  auto rm_off = [&](uint32_t q) {
    const uint32_t row = fdiv(q, a.units_per_row);
    const uint32_t col = q - row * a.units_per_row.d;
    return (int64_t)row * a.ld_bytes + (int64_t)col * 16;
  };
  auto load = [&](uint32_t base, u32x4* v) {
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const uint32_t q = base + threadIdx.x + u * 256u;
      if (q < a.units_per_block) {
        if (UNPACK)
          v[u] = ld<true>(reinterpret_cast<const u32x4*>(a.ccl + strip_base + (int64_t)q * 16));
        else
          v[u] = ld<true>(reinterpret_cast<const u32x4*>(src_rm + rm_off(q)));
      }
    }
  };
  auto store = [&](uint32_t base, const u32x4* v) {
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const uint32_t q = base + threadIdx.x + u * 256u;
      if (q < a.units_per_block) {
        if (UNPACK)
          *reinterpret_cast<u32x4*>(dst_rm + rm_off(q)) = v[u];
        else
          *reinterpret_cast<u32x4*>(a.ccl_out + strip_base + (int64_t)q * 16) = v[u];
      }
    }
  };
  uint32_t base = blockIdx.x * kRound;
  if (base >= a.units_per_block) return;
  u32x4 cur[UNROLL], nxt[UNROLL];
  load(base, cur);
  for (; base < a.units_per_block; base += stride) {
    const uint32_t next = base + stride;
    if (next < a.units_per_block) load(next, nxt);
    store(base, cur);
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) cur[u] = nxt[u];
  }
}

// Stored-transpose pack through LDS, for blocks whose sides are multiples of
// 64 but not of the register kernel's block edge below (fp8 blocks with a
// side of 64 mod 128): src holds X^T (cols x rows, leading dimension ld
// elements), X is rows x cols of element type E. A 64 x 64 tile is read
// along X's rows (contiguous in src) in 16-byte chunks, transposed through
// LDS and written in 16-byte chunks along X's columns (contiguous in the
// CCL strip). Tiles never straddle blocks (hr, wc multiples of 64).
struct TransArgs {
  const char* src;
  char* dst;
  int64_t ld;              // elements
  int64_t strip;           // bytes
  int64_t hr, wc;          // elements
  int32_t grid_c;
};

template <typename E>
__global__ void __launch_bounds__(256) pack_trans_kernel(TransArgs a) {
  constexpr int EPC = 16 / sizeof(E);                  // elements per 16-byte chunk
  constexpr int CPR = 64 / EPC;                        // chunks per 64-element row
  constexpr int ITER = 64 * CPR / 256;                 // chunks per thread
  __shared__ E tile[64][64 + 16 / sizeof(E)];
  const int64_t r0 = (int64_t)blockIdx.y * 64;        // X rows = src columns
  const int64_t c0 = (int64_t)blockIdx.x * 64;        // X cols = src rows
  const int t = threadIdx.x;
  const E* src = reinterpret_cast<const E*>(a.src);
#pragma unroll
  for (int i = 0; i < ITER; ++i) {
    const int idx = t + i * 256;
    const int sr = idx / CPR, ch = idx % CPR;
    uint4 v = *reinterpret_cast<const uint4*>(src + (c0 + sr) * a.ld + r0 + ch * EPC);
    const E* e = reinterpret_cast<const E*>(&v);
#pragma unroll
    for (int j = 0; j < EPC; ++j) tile[sr][ch * EPC + j] = e[j];
  }
  __syncthreads();
  const int64_t pr = r0 / a.hr, pc = c0 / a.wc;
  const int64_t b = pr * a.grid_c + pc;
  E* strip = reinterpret_cast<E*>(a.dst + b * a.strip);
  const int64_t rl0 = r0 - pr * a.hr, cl0 = c0 - pc * a.wc;
#pragma unroll
  for (int i = 0; i < ITER; ++i) {
    const int idx = t + i * 256;
    const int xr = idx / CPR, ch = idx % CPR;
    uint4 v;
    E* e = reinterpret_cast<E*>(&v);
#pragma unroll
    for (int j = 0; j < EPC; ++j) e[j] = tile[ch * EPC + j][xr];
    *reinterpret_cast<uint4*>(strip + (rl0 + xr) * a.wc + cl0 + ch * EPC) = v;
  }
}

// Stored-transpose pack without LDS. With EPC elements per 16-byte chunk,
// each thread moves an EPC x EPC block: it reads EPC chunks, one from each
// of EPC consecutive rows of the stored transpose, transposes the block in
// registers (byte permutes) and writes EPC chunks along consecutive rows of
// the CCL strip. Lane (a, b) = (lane % 8, lane / 8) covers X rows
// R0 + EPC a .. + EPC - 1 and X columns C0 + EPC b .. + EPC - 1, so a wave
// covers a WB x WB block (WB = 8 EPC) and each of its loads and stores
// touches 8 rows x 128 contiguous bytes. The 4 waves of a workgroup take 4
// consecutive blocks along X's columns. Blocks never straddle CCL blocks
// (hr and wc are multiples of WB). NTL: streaming loads (sources beyond the
// Infinity Cache). The stores always stream: on a 134 MB transpose that
// measured +12 % from HBM and no loss with the source cache-resident.
template <typename E, bool NTL>
__global__ void __launch_bounds__(256) pack_trans_reg_kernel(TransArgs a, int32_t wb_cols) {
  constexpr int EPC = 16 / (int)sizeof(E);
  constexpr int WB = 8 * EPC;
  typedef E ev __attribute__((ext_vector_type(EPC)));
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  // Row block by of column group bx: blockIdx.y skewed by 2 blocks per
  // column group, so that the workgroups resident at one time read chunks
  // spread over the width of the stored rows instead of one 8 KiB band of
  // them (a bijection for each bx). Measured from HBM against no skew:
  // 134 MB X^T 0.663-0.666 of 8 TB/s against 0.627-0.628, 470 MB W_up^T
  // 0.710 against 0.698-0.699; skews of 1, 3 and 4 were 0-1 % slower, 8
  // and 16 (several column groups then share a band) 4 % and 20 % slower.
  const int32_t bx = blockIdx.x, by = (int32_t)((blockIdx.y + blockIdx.x * 2u) % gridDim.y);
  const int32_t wcb = bx * 4 + wave;
  if (wcb >= wb_cols) return;
  const int la = lane & 7, lb = lane >> 3;
  const int64_t R0 = (int64_t)by * WB, C0 = (int64_t)wcb * WB;
  const E* src = reinterpret_cast<const E*>(a.src) + (C0 + EPC * lb) * a.ld + R0 + EPC * la;
  ev in[EPC];
#pragma unroll
  for (int j = 0; j < EPC; ++j)
    in[j] = __builtin_bit_cast(ev, ld<NTL>(reinterpret_cast<const u32x4*>(src + j * a.ld)));
  const int32_t pr = (int32_t)(R0 / a.hr), pc = (int32_t)(C0 / a.wc);
  E* strip = reinterpret_cast<E*>(a.dst + ((int64_t)pr * a.grid_c + pc) * a.strip);
  E* dst = strip + (R0 - pr * a.hr + EPC * la) * a.wc + (C0 - pc * a.wc) + EPC * lb;
#pragma unroll
  for (int i = 0; i < EPC; ++i) {
    ev o;
#pragma unroll
    for (int j = 0; j < EPC; ++j) o[j] = in[j][i];
    st<true>(reinterpret_cast<u32x4*>(dst + i * a.wc), __builtin_bit_cast(u32x4, o));
  }
}

// Any shape: one element per thread, src holds X^T.
template <typename E>
__global__ void __launch_bounds__(256) pack_trans_scalar_kernel(TransArgs a, int64_t rows,
                                                                int64_t cols) {
  const int64_t n = rows * cols;
  const E* src = reinterpret_cast<const E*>(a.src);
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const int64_t r = i / cols, c = i % cols;          // write order: along X rows
    const int64_t pr = r / a.hr, pc = c / a.wc;
    const int64_t b = pr * a.grid_c + pc;
    E* strip = reinterpret_cast<E*>(a.dst + b * a.strip);
    strip[(r - pr * a.hr) * a.wc + (c - pc * a.wc)] = src[c * a.ld + r];
  }
}

int grid_x_for(uint32_t units, int unroll) {
  uint64_t wgs = ((uint64_t)units + 256ull * unroll - 1) / (256ull * unroll);
  if (wgs > 4096) wgs = 4096;
  return (int)(wgs ? wgs : 1);
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

template <typename U>
void copy_launch(dim3 grid, const PackArgs& a, bool unpack, hipStream_t stream) {
  if (unpack)
    hipLaunchKernelGGL((copy_kernel<U, true, false, false>), grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL((copy_kernel<U, false, false, false>), grid, dim3(256), 0, stream, a);
}

// path 2: register blocks, 1: LDS tiles, 0: one element per thread.
template <typename E>
void trans_launch(const Layout& L, const TransArgs& a, int path, bool ntl, hipStream_t stream) {
  if (path == 2) {
    constexpr int WB = 8 * 16 / (int)sizeof(E);
    const int32_t wb_cols = (int32_t)(L.cols / WB);
    dim3 grid((unsigned)((wb_cols + 3) / 4), (unsigned)(L.rows / WB));
    if (ntl)
      hipLaunchKernelGGL((pack_trans_reg_kernel<E, true>), grid, dim3(256), 0, stream, a, wb_cols);
    else
      hipLaunchKernelGGL((pack_trans_reg_kernel<E, false>), grid, dim3(256), 0, stream, a, wb_cols);
  } else if (path == 1) {
    dim3 grid((unsigned)(L.cols / 64), (unsigned)(L.rows / 64));
    hipLaunchKernelGGL((pack_trans_kernel<E>), grid, dim3(256), 0, stream, a);
  } else {
    int64_t n = L.rows * L.cols;
    int64_t wgs = (n + 255) / 256;
    if (wgs > 8192) wgs = 8192;
    hipLaunchKernelGGL((pack_trans_scalar_kernel<E>), dim3((unsigned)wgs), dim3(256), 0, stream, a,
                       L.rows, L.cols);
  }
}

}  // namespace

hipError_t launch_copy(const Plan& p, int op, const void* rowmajor, int64_t ld, void* ccl_buf,
                       bool unpack, hipStream_t stream) {
  const Layout& L = p.lay[op];
  const int64_t e = L.elem_bytes;
  const int64_t row_bytes = L.block_cols * e;
  const bool vec = (row_bytes % 16 == 0) && ((ld * e) % 16 == 0) && aligned16(rowmajor) &&
                   aligned16(ccl_buf) && (L.strip_stride_bytes % 16 == 0);
  const int64_t unit = vec ? 16 : e;
  PackArgs a;
  a.rm = static_cast<const char*>(rowmajor);
  a.rm_out = const_cast<char*>(static_cast<const char*>(rowmajor));
  a.ccl = static_cast<const char*>(ccl_buf);
  a.ccl_out = static_cast<char*>(ccl_buf);
  a.ld_bytes = ld * e;
  a.strip = L.strip_stride_bytes;
  a.hr = L.block_rows;
  a.row_bytes = row_bytes;
  a.grid_c = (int32_t)L.grid_c;
  a.units_per_block = (uint32_t)(L.block_rows * row_bytes / unit);
  a.units_per_row = make_div((uint32_t)(row_bytes / unit));
  const unsigned strips = (unsigned)(L.grid_r * L.grid_c);
  dim3 grid(grid_x_for(a.units_per_block, 4), strips);
  if (vec) {
    const bool big = L.rows * L.cols * e > kInfinityCacheBytes;
    if (big) {
      // above the cache size both sides stream (measured: +10 % on 470 MB)
      if (unpack)
        hipLaunchKernelGGL((copy_kernel<u32x4, true, true, true>), grid, dim3(256), 0, stream, a);
      else
        hipLaunchKernelGGL((copy_kernel<u32x4, false, true, true>), grid, dim3(256), 0, stream, a);
    } else {
      // resident grid: kResidentWgs workgroups in all, at most one round each per strip
      const unsigned per_strip = std::max(1u, kResidentWgs / strips);
      const dim3 g((unsigned)std::min<int64_t>(per_strip, grid.x), strips);
      if (unpack)
        hipLaunchKernelGGL((copy_stream_kernel<true>), g, dim3(256), 0, stream, a);
      else
        hipLaunchKernelGGL((copy_stream_kernel<false>), g, dim3(256), 0, stream, a);
    }
  } else if (e == 1) {
    copy_launch<uint8_t>(grid, a, unpack, stream);
  } else if (e == 2) {
    copy_launch<uint16_t>(grid, a, unpack, stream);
  } else {
    copy_launch<uint32_t>(grid, a, unpack, stream);
  }
  return hipGetLastError();
}

hipError_t launch_pack_trans(const Plan& p, int op, const void* src, int64_t ld, void* dst,
                             hipStream_t stream) {
  const Layout& L = p.lay[op];
  const int64_t e = L.elem_bytes;
  TransArgs a;
  a.src = static_cast<const char*>(src);
  a.dst = static_cast<char*>(dst);
  a.ld = ld;
  a.strip = L.strip_stride_bytes;
  a.hr = L.block_rows;
  a.wc = L.block_cols;
  a.grid_c = (int32_t)L.grid_c;
  const bool vec = (ld * e) % 16 == 0 && aligned16(src) && aligned16(dst) &&
                   L.strip_stride_bytes % 16 == 0;
  const int64_t wb = 8 * 16 / e;      // block edge of the register-transpose kernel
  int path = 0;
  if (vec && L.block_rows % wb == 0 && L.block_cols % wb == 0 && L.rows / wb <= 65535)
    path = 2;
  else if (vec && L.block_rows % 64 == 0 && L.block_cols % 64 == 0 && L.rows / 64 <= 65535)
    path = 1;
  // Loads stream at every size: the stored tensor is read once (measured on
  // the 134 MB X^T from HBM: 5.05 against 4.92 TB/s).
  const bool ntl = true;
  if (e == 1)
    trans_launch<uint8_t>(L, a, path, ntl, stream);
  else if (e == 2)
    trans_launch<uint16_t>(L, a, path, ntl, stream);
  else
    trans_launch<uint32_t>(L, a, path, ntl, stream);
  return hipGetLastError();
}

}  // namespace ccl
