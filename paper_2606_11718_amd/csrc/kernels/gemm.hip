// C = A B on CCL operands for gfx950 (Sec. II-B, III-C: the arithmetic is
// the plain tiled GEMM; only the operand address map is CCL's).
//
// Workgroup = 4 waves (2 x 2), output tile BM x BN, K step 64.
//  * Workgroup -> tile: tile_map.hpp. Dispatch is round-robin over the 8
//    XCDs, so the map sends every tile to an XCD of the chiplet that owns
//    it (Sec. III-A).
//  * Operand addressing: inside one CCL block an operand is row-major with
//    leading dimension wc; A changes block every K/Gc columns and B every
//    K/Gr rows, which a K step (64) never straddles. The same descriptor
//    also expresses plain row-major operands.
//  * Global -> LDS: direct-to-LDS 16-byte loads (global_load_lds_dwordx4),
//    two LDS stages; the next K step is in flight while MFMAs run on the
//    current one. Which 16-byte chunk each lane fetches is permuted (XOR
//    swizzle) so the fragment reads below hit distinct LDS banks.
//  * A (K contiguous) fragments: ds_read_b128. B (N contiguous) fragments:
//    ds_read_b64_tr_b16, which transposes 16-bit data across each group of
//    16 lanes (lane l, element j <- lane 4j + l/4, element l%4).
//  * Matrix cores: v_mfma_f32_32x32x16_bf16 with fp32 accumulators; the
//    product is formed as C^T tiles so that each lane ends up holding four
//    consecutive columns of C, written as one 8-byte store (bf16, RNE).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.hpp"

namespace ccl {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;

constexpr int kBK = 64;
constexpr int kThreads = 256;

struct GemmParams {
  const uint16_t* A;
  const uint16_t* B;
  uint16_t* C;
  OperandAddr a, b, c;
  TileMap map;
  int32_t ksteps;       // K / 64
  int32_t remap;        // 1: XCD-aware map; 0: native raster over the whole C
  int32_t grid_r;       // Gr (native raster)
};

// LDS chunk swizzles (16-byte chunk index XOR a function of the row).
// A rows are 128 B (8 chunks): rows r..r+15 read at one logical chunk land
// on 16 distinct (row parity, slot) pairs.
__device__ __forceinline__ int swz_a(int row) { return (row & 7) ^ ((row >> 3) & 1); }
// B rows are BN*2 bytes: the 4 rows one 16-lane transpose read touches get
// disjoint 32-byte (and 64-byte) bank windows.
__device__ __forceinline__ int swz_b(int row) { return ((row & 3) << 1) ^ ((row & 3) << 2); }

__device__ __forceinline__ uint32_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

template <int BM, int BN>
struct Tile {
  static constexpr int WM = BM / 2, WN = BN / 2;       // wave tile
  static constexpr int TM = WM / 32, TN = WN / 32;     // MFMA tiles per wave
  static constexpr int A_BYTES = BM * kBK * 2;
  static constexpr int B_BYTES = kBK * BN * 2;
  static constexpr int NA = BM / 32;                   // A load instructions per wave per stage
  static constexpr int CPR_B = BN / 8;                 // 16-byte chunks per B row
  static constexpr int RPI_B = 64 / CPR_B;             // B rows per load instruction
  static constexpr int NB = BN / 32;                   // B load instructions per wave per stage
};

// MFMA operand fragments of one kk sub-step: A rows and B columns.
template <int TM, int TN>
struct FragSet {
  bf16x8 a[TM];
  bf16x8 b[TN];
};

// Instruction classes for __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedMfma = 0x008;
constexpr int kSchedVmemRead = 0x020;
constexpr int kSchedDsRead = 0x100;

template <int BM, int BN>
__global__ void __launch_bounds__(kThreads, 1) gemm_kernel(GemmParams p) {
  // The host pass only needs the launch stub; the body uses device-only
  // buffer-resource builtins.
#if defined(__HIP_DEVICE_COMPILE__)
  using T = Tile<BM, BN>;
  __shared__ __attribute__((aligned(1024))) char smA0[T::A_BYTES];
  __shared__ __attribute__((aligned(1024))) char smA1[T::A_BYTES];
  __shared__ __attribute__((aligned(1024))) char smB0[T::B_BYTES];
  __shared__ __attribute__((aligned(1024))) char smB1[T::B_BYTES];

  int32_t pr, pc, ti, tj;
  if (p.remap) {
    if (!map_tile(p.map, blockIdx.x, &pr, &pc, &ti, &tj)) return;
  } else {
    // native order: grouped raster over the whole tile grid, XCD-oblivious
    const int32_t TMg = p.map.tiles_m * p.grid_r, TNg = p.map.tiles_n * p.map.grid_c;
    const int32_t t = blockIdx.x;
    if (t >= TMg * TNg) return;
    const int32_t per_group = p.map.group_m * TNg;
    const int32_t grp = t / per_group, first = grp * p.map.group_m;
    const int32_t gm = min(p.map.group_m, TMg - first);
    const int32_t w = t - grp * per_group;
    const int32_t tig = first + w % gm, tjg = w / gm;
    pr = tig / p.map.tiles_m;
    ti = tig - pr * p.map.tiles_m;
    pc = tjg / p.map.tiles_n;
    tj = tjg - pc * p.map.tiles_n;
  }

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  // ---- global -> LDS: per-lane byte offsets from the K step's tile corner ----
  uint32_t a_voff[T::NA];
#pragma unroll
  for (int i = 0; i < T::NA; ++i) {
    const int row = 8 * (wave * T::NA + i) + (lane >> 3);
    const int chunk = (lane & 7) ^ swz_a(row);
    a_voff[i] = (uint32_t)(row * p.a.ld + chunk * 8) * 2u;
  }
  uint32_t b_voff[T::NB];
#pragma unroll
  for (int i = 0; i < T::NB; ++i) {
    const int row = T::RPI_B * (wave * T::NB + i) + lane / T::CPR_B;
    const int chunk = (lane % T::CPR_B) ^ swz_b(row);
    b_voff[i] = (uint32_t)(row * p.b.ld + chunk * 8) * 2u;
  }
  // Bytes a K step may touch from its corner: loads outside return zero.
  const int32_t a_extent = (BM - 1) * p.a.ld * 2 + kBK * 2;
  const int32_t b_extent = (kBK - 1) * p.b.ld * 2 + BN * 2;

  // ---- LDS fragment read offsets (bytes) ----
  int32_t a_rd[4];
  {
    const int row = wm * T::WM + (lane & 31);
    const int h = lane >> 5;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) a_rd[kk] = row * 128 + (((2 * kk + h) ^ swz_a(row)) * 16);
  }
  int32_t b_rd[T::TN][2];
  {
    const int g = lane >> 4, s = lane & 15;
#pragma unroll
    for (int nt = 0; nt < T::TN; ++nt) {
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int krow = 8 * (g >> 1) + 4 * r + (s >> 2);
        const int col = wn * T::WN + nt * 32 + 16 * (g & 1) + 4 * (s & 3);
        b_rd[nt][r] = krow * (BN * 2) + (((col >> 3) ^ swz_b(krow)) * 16) + ((col >> 2) & 1) * 8;
      }
    }
  }

  // ---- operand corners; K-slice block advances every kslice columns/rows ----
  const uint16_t* a_base = p.A + pr * p.a.part + (int64_t)(ti * BM) * p.a.ld;
  const uint16_t* b_base = p.B + pc * p.b.part + tj * BN;
  int64_t a_slice_off = 0, b_slice_off = 0;
  int32_t a_kl = 0, b_kl = 0;

  // Issue the direct-to-LDS loads of the next K step. With live == false
  // the descriptors cover zero bytes: every load is out of range, touches
  // no memory and writes zeros to the (unused) stage.
  auto load_stage = [&](char* smA, char* smB, bool live) {
    const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(a_base + a_slice_off + a_kl), (short)0, live ? a_extent : 0, 0x00020000);
    const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(b_base + b_slice_off + (int64_t)b_kl * p.b.ld), (short)0, live ? b_extent : 0,
        0x00020000);
#pragma unroll
    for (int i = 0; i < T::NA; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void*)(smA + (wave * T::NA + i) * 1024), 16,
                                               a_voff[i], 0, 0, 0);
#pragma unroll
    for (int i = 0; i < T::NB; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void*)(smB + (wave * T::NB + i) * 1024), 16,
                                               b_voff[i], 0, 0, 0);
    // advance to the next K step (branch-free; past the last step the
    // corners are never used with a non-empty descriptor)
    a_kl += kBK;
    const bool a_wrap = a_kl == p.a.kslice;
    a_kl = a_wrap ? 0 : a_kl;
    a_slice_off += a_wrap ? p.a.slice : 0;
    b_kl += kBK;
    const bool b_wrap = b_kl == p.b.kslice;
    b_kl = b_wrap ? 0 : b_kl;
    b_slice_off += b_wrap ? p.b.slice : 0;
  };

  using Frags = FragSet<T::TM, T::TN>;
  auto read_frags = [&](const char* smA, const char* smB, int kk, Frags& f) {
#pragma unroll
    for (int mt = 0; mt < T::TM; ++mt)
      f.a[mt] = *(const lds_bf16x8*)(smA + a_rd[kk] + mt * 32 * 128);
#pragma unroll
    for (int nt = 0; nt < T::TN; ++nt) {
      i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (lds_i16x4*)(smB + b_rd[nt][0] + kk * 16 * BN * 2));
      i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (lds_i16x4*)(smB + b_rd[nt][1] + kk * 16 * BN * 2));
      f.b[nt] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    }
  };

  f32x16 acc[T::TM][T::TN];
#pragma unroll
  for (int i = 0; i < T::TM; ++i)
#pragma unroll
    for (int j = 0; j < T::TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  auto mfmas = [&](const Frags& f) {
#pragma unroll
    for (int mt = 0; mt < T::TM; ++mt)
#pragma unroll
      for (int nt = 0; nt < T::TN; ++nt)
        acc[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.b[nt], f.a[mt], acc[mt][nt], 0, 0, 0);
  };

  constexpr int kMfmaPerKK = T::TM * T::TN;
  constexpr int kReadsPerKK = T::TM + 2 * T::TN;
  // Behind each MFMA issue at most one buffer load and one LDS read, so the
  // matrix pipe stays fed while the memory instructions drain.
  auto interleave = [&](int n_vmem) {
#pragma unroll
    for (int i = 0; i < kMfmaPerKK; ++i) {
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
      if (i < n_vmem) __builtin_amdgcn_sched_group_barrier(kSchedVmemRead, 1, 0);
      if (i < kReadsPerKK) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
    }
#pragma unroll
    for (int i = kMfmaPerKK; i < n_vmem; ++i) __builtin_amdgcn_sched_group_barrier(kSchedVmemRead, 1, 0);
#pragma unroll
    for (int i = kMfmaPerKK; i < kReadsPerKK; ++i) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
    __builtin_amdgcn_sched_barrier(0);
  };

  Frags f0, f1;
  // One K step on LDS stage (smA, smB), whose kk = 0 fragments are in f0.
  // The next step's loads go to (nA, nB) (dummy when !live) and its kk = 0
  // fragments are read into f0 at the end.
  auto step = [&](const char* smA, const char* smB, char* nA, char* nB, bool live) {
    load_stage(nA, nB, live);
    read_frags(smA, smB, 1, f1);
    mfmas(f0);
    interleave(T::NA + T::NB);
    read_frags(smA, smB, 2, f0);
    mfmas(f1);
    interleave(0);
    read_frags(smA, smB, 3, f1);
    mfmas(f0);
    interleave(0);
    // all of this stage is in registers; the next stage's loads must land
    wait_vm_all();
    __syncthreads();
    read_frags(nA, nB, 0, f0);
    mfmas(f1);
    interleave(0);
  };

  const int32_t ksteps = p.ksteps;
  load_stage(smA0, smB0, true);
  wait_vm_all();
  __syncthreads();
  read_frags(smA0, smB0, 0, f0);
  for (int32_t s = 0; s < ksteps; s += 2) {
    step(smA0, smB0, smA1, smB1, s + 1 < ksteps);
    if (s + 1 < ksteps) step(smA1, smB1, smA0, smB0, s + 2 < ksteps);
  }

  // ---- epilogue: lane holds C[m][n .. n+3] for each (mt, nt, q) ----
  uint16_t* c_tile = p.C + pr * p.c.part + pc * p.c.slice + (int64_t)(ti * BM) * p.c.ld + tj * BN;
#pragma unroll
  for (int mt = 0; mt < T::TM; ++mt) {
    const int m = wm * T::WM + mt * 32 + (lane & 31);
#pragma unroll
    for (int nt = 0; nt < T::TN; ++nt) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = wn * T::WN + nt * 32 + 8 * q + 4 * (lane >> 5);
        uint2 v;
        v.x = bf16_rne(acc[mt][nt][4 * q + 0]) | (bf16_rne(acc[mt][nt][4 * q + 1]) << 16);
        v.y = bf16_rne(acc[mt][nt][4 * q + 2]) | (bf16_rne(acc[mt][nt][4 * q + 3]) << 16);
        *reinterpret_cast<uint2*>(c_tile + (int64_t)m * p.c.ld + n) = v;
      }
    }
  }
#endif
}

// Records, per workgroup of the GEMM grid, the XCD it ran on and its tile.
__global__ void __launch_bounds__(64) dispatch_probe_kernel(TileMap map, int32_t tiles_m,
                                                            int32_t tiles_n, int32_t* out) {
  if (threadIdx.x != 0) return;
  uint32_t xcc;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
  int32_t pr, pc, ti, tj;
  int32_t* o = out + 4 * (int64_t)blockIdx.x;
  o[0] = (int32_t)(xcc & 0xf);
  if (map_tile(map, blockIdx.x, &pr, &pc, &ti, &tj)) {
    o[1] = pr * tiles_m + ti;
    o[2] = pc * tiles_n + tj;
    o[3] = pr * map.grid_c + pc;
  } else {
    o[1] = o[2] = o[3] = -1;
  }
}

}  // namespace

hipError_t launch_gemm(const Plan& p, const void* A, const void* B, void* C,
                       const OperandAddr& a, const OperandAddr& b, const OperandAddr& c,
                       bool remap, hipStream_t stream) {
  const GemmConfig& g = p.gemm;
  GemmParams gp;
  gp.A = static_cast<const uint16_t*>(A);
  gp.B = static_cast<const uint16_t*>(B);
  gp.C = static_cast<uint16_t*>(C);
  gp.a = a;
  gp.b = b;
  gp.c = c;
  gp.map = tile_map(p);
  gp.ksteps = (int32_t)(p.K / kBK);
  gp.remap = remap ? 1 : 0;
  gp.grid_r = p.Gr;
  const unsigned wgs = remap ? (unsigned)g.workgroups
                             : (unsigned)(g.tiles_m * g.tiles_n * p.G);
  dim3 grid(wgs), block(kThreads);
  if (g.tile_m == 256 && g.tile_n == 256)
    hipLaunchKernelGGL((gemm_kernel<256, 256>), grid, block, 0, stream, gp);
  else if (g.tile_m == 256 && g.tile_n == 128)
    hipLaunchKernelGGL((gemm_kernel<256, 128>), grid, block, 0, stream, gp);
  else if (g.tile_m == 128 && g.tile_n == 256)
    hipLaunchKernelGGL((gemm_kernel<128, 256>), grid, block, 0, stream, gp);
  else if (g.tile_m == 128 && g.tile_n == 128)
    hipLaunchKernelGGL((gemm_kernel<128, 128>), grid, block, 0, stream, gp);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_dispatch_probe(const Plan& p, int32_t* out, hipStream_t stream) {
  hipLaunchKernelGGL(dispatch_probe_kernel, dim3((unsigned)p.gemm.workgroups), dim3(64), 0, stream,
                     tile_map(p), (int32_t)p.gemm.tiles_m, (int32_t)p.gemm.tiles_n, out);
  return hipGetLastError();
}

}  // namespace ccl
