// C = A B (or alpha A B + beta C) on CCL operands for gfx950 (Sec. II-B,
// III-C: the arithmetic is the plain tiled GEMM; only the operand address
// map is CCL's).
//
// The kernels share the tile map, the operand descriptors, the
// direct-to-LDS loads and the epilogue:
//  * gemm_kernel: bf16 operands (described below);
//  * gemm_a2_kernel: bf16 256x256 with A staged in 64-K pairs of steps
//    (whole-line A loads), otherwise gemm_kernel's schedule;
//  * gemm_k64_kernel: bf16 tiles below 256x256 with 64-K stages;
//  * gemm_fp8p_kernel: fp8 operands on 256x256 tiles with 8 waves and K
//    blocks that are multiples of 128 (v_mfma_f32_16x16x128_f8f6f4), the
//    fragment reads pipelined across steps;
//  * gemm_fp8x_kernel: the same plans with two stages and the fragment reads
//    after each step's barrier (CCL_GEMM_FP8_PIPE=0);
//  * gemm_fp8_kernel: the other fp8 plans (v_mfma_f32_32x32x64_f8f6f4).
//
// bf16: workgroup = 2 x WGN waves, output tile BM x BN, K step 32 (kBK).
//  * Workgroup -> tile: tile_map.hpp. Dispatch is round-robin over the 8
//    XCDs, so the map sends every tile to an XCD of the chiplet that owns
//    it (Sec. III-A).
//  * Operand addressing: inside one CCL block an operand is row-major with
//    leading dimension wc; A changes block every K/Gc columns and B every
//    K/Gr rows, which a K step never straddles. The same descriptor also
//    expresses plain row-major operands.
//  * Global -> LDS: direct-to-LDS 16-byte buffer loads, four LDS stages; the
//    loads of step s+3 are issued while the MFMAs of step s run. Which
//    16-byte chunk each lane fetches is permuted (XOR swizzle) so the
//    fragment reads below hit distinct LDS banks.
//  * A (K contiguous) fragments: ds_read_b128. B (N contiguous) fragments:
//    ds_read_b64_tr_b16, which transposes 16-bit data across each group of
//    16 lanes (lane l, element j <- lane 4j + l/4, element l%4).
//  * Matrix cores: v_mfma_f32_16x16x32_bf16 with fp32 accumulators (one
//    instruction covers a whole K step). Measured on MI355X with random
//    operands, this shape does about 12 % more work per joule than
//    32x32x16, which is what counts when the GEMM runs at the socket power
//    limit. The product is formed as C^T tiles so that each lane ends up
//    holding four consecutive columns of C, written as one 8-byte store
//    (bf16, RNE).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <type_traits>

#include "kernels.hpp"

namespace ccl {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;

constexpr int kBK = 32;          // K extent of one main-loop step
constexpr int kStages = 4;       // fp8 LDS stages; loads run kStages-1 steps ahead
// bf16 LDS stages (32 KiB each for a 256x256 tile); loads run kStagesBf16-1
// steps ahead.
#ifndef CCL_BF16_STAGES
#define CCL_BF16_STAGES 4
#endif
constexpr int kStagesBf16 = CCL_BF16_STAGES;

struct GemmParams {
  const uint16_t* A;
  const uint16_t* B;
  void* C;                // bf16, or fp32 when c_f32
  OperandAddr a, b, c;
  TileMap map;
  int32_t ksteps;       // K / (the kernel's K step)
  int32_t remap;        // 1: XCD-aware map; 0: native raster over the whole C
  int32_t grid_r;       // Gr (native raster)
  int32_t epi;          // epilogue: 0 acc, 1 alpha*acc, 2 alpha*acc + beta*C (C read)
  int32_t c_f32;        // C elements are fp32 (else bf16)
  float alpha, beta;
  int32_t ksteps_per_split;  // K steps of one split (= ksteps without split-K)
  int32_t round_fast;   // bf16: K blocks and split starts are 4-step aligned (rounds path)
  int32_t splits_total; // split-K ranges per tile (reduce kernel)
  float* ws;            // split-K: fp32 partial tiles (null: write C directly)
  uint64_t* timeline;   // bf16 kernel: kTimelineWords per wave (null: not recorded)
};

// LDS chunk swizzles (16-byte chunk index XOR a function of the row).
// Bank model of gfx950, measured with SQ_LDS_BANK_CONFLICT on single-lane
// pairs: 64 banks of 4 bytes; an 8-byte read (ds_read_b64, also the
// transposing form) serves each half-wave in one cycle; ds_read_b128 serves
// a half-wave in two cycles, split by the parity of lane bits 2..4 (lanes
// 0-3, 12-15, 20-23, 24-27 together). A read is conflict-free when the
// lanes of each such group touch distinct banks.
//
// A rows are 64 B (4 chunks). swz_a serves the fp8 kernel's A reads (32
// rows x 2 chunks per half-wave): chunk XOR (row / 4) mod 4. swz_a16 serves
// the bf16 kernel's 16x16 A reads (16 rows x 4 chunks per wave): chunk XOR
// 2 * (bit 2 of row). Both measure zero conflicts.
__device__ __forceinline__ int swz_a(int row) { return (row >> 2) & 3; }
__device__ __forceinline__ int swz_a16(int row) { return ((row >> 2) & 1) << 1; }
// B rows are BN*2 bytes (16 or 32 chunks). The 32 lanes of a half-wave of
// one bf16 transposed fragment read touch 8 rows (k = 8g + 4r + j for two
// neighbouring g, j = 0..3) x 2 neighbouring chunks; XOR-ing the chunk with
// 2 * ((row & 3) | (row & 8) >> 1) sends these 16 (row, chunk) pairs to 16
// distinct 16-byte bank slots.
__device__ __forceinline__ int swz_b(int row) { return ((row & 3) << 1) | (((row >> 3) & 1) << 3); }

__device__ __forceinline__ uint32_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char lds_char;

// Raw buffer descriptor (stride 0): `num_records` bytes from `base`; a load
// at offset >= num_records returns zero without touching memory.
__device__ __forceinline__ i32x4 buffer_rsrc(const void* base, int32_t num_records) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  i32x4 r;
  r[0] = (int)(uint32_t)a;
  r[1] = (int)((a >> 32) & 0xffffu);
  r[2] = num_records;
  r[3] = 0x00020000;
  return r;
}

// 16 bytes per lane from the buffer straight into LDS at `lds` + 16*lane.
// Written as inline assembly so that the compiler does not track these LDS
// writes itself: it cannot tell the stage arrays apart and would wait for
// loads of later stages before reading the current one. The kernel orders
// them with explicit vmcnt waits and barriers; nothing else in it uses M0.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_dma16(i32x4 rsrc, uint32_t voff, const char* lds) {
  const uint32_t m0v = (uint32_t)(uintptr_t)(const lds_char*)lds;
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :: "s"(m0v), "v"(voff), "s"(rsrc) : "m0");
}
// The same with a scalar byte offset added to the memory address (the LDS
// destination is unchanged).
__device__ __forceinline__ void lds_dma16_so(i32x4 rsrc, uint32_t voff, uint32_t soff, const char* lds) {
  const uint32_t m0v = (uint32_t)(uintptr_t)(const lds_char*)lds;
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :: "s"(m0v), "v"(voff), "s"(rsrc), "s"(soff) : "m0");
}
// A run of loads that share one M0: the first sets M0 to the LDS
// destination of the run, the next ones (lds_dma16_next<OFF>) reuse it.
// Their instruction offset moves both the memory address and the LDS
// destination by OFF bytes (the scalar offset moves the memory address
// only), so load i of a run lands OFF = 1024 i bytes after the first when
// its per-lane offset is the plain one minus OFF. The run's loads are
// volatile asm, kept in order, and nothing between them writes M0.
__device__ __forceinline__ void lds_dma16_first(i32x4 rsrc, uint32_t voff, uint32_t soff,
                                                const char* lds) {
  const uint32_t m0v = (uint32_t)(uintptr_t)(const lds_char*)lds;
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :: "s"(m0v), "v"(voff), "s"(rsrc), "s"(soff) : "m0");
}
template <int OFF>
__device__ __forceinline__ void lds_dma16_next(i32x4 rsrc, uint32_t voff, uint32_t soff) {
  static_assert(OFF > 0 && OFF < 4096, "12-bit instruction offset");
  asm volatile("buffer_load_dwordx4 %0, %1, %2 offen offset:%3 lds"
               :: "v"(voff), "s"(rsrc), "s"(soff), "n"(OFF));
}
#pragma clang diagnostic pop

// s_waitcnt immediate: vmcnt(vm) and lgkmcnt(lgkm), expcnt not waited on.
constexpr int waitcnt_imm(int vm, int lgkm) {
  return (vm & 15) | (7 << 4) | ((lgkm & 15) << 8) | (((vm >> 4) & 3) << 14);
}

// Output tile BM x BN computed by a 2 x WGN grid of waves, 16 x 16 MFMA
// tiles.
template <int BM, int BN, int WGN>
struct Tile {
  static constexpr int NW = 2 * WGN;                   // waves per workgroup
  static constexpr int THREADS = 64 * NW;
  static constexpr int WM = BM / 2, WN = BN / WGN;     // wave tile
  static constexpr int TM = WM / 16, TN = WN / 16;     // MFMA tiles per wave
  static constexpr int A_BYTES = BM * kBK * 2;         // one stage
  static constexpr int B_BYTES = kBK * BN * 2;
  static constexpr int NA = BM / (16 * NW);            // A loads per wave per stage (1 KB each)
  static constexpr int CPR_B = BN / 8;                 // 16-byte chunks per B row
  static constexpr int RPI_B = 64 / CPR_B;             // B rows per load instruction
  static constexpr int NB = BN / (16 * NW);            // B loads per wave per stage
  static constexpr int NL = NA + NB;
  static_assert(NA >= 1 && NB >= 1 && TN >= 1, "tile too small for the wave grid");
  static_assert(TM % 2 == 0, "the step splits the A fragments in two halves");
  static_assert(TM * TN * 4 <= 256, "accumulators must fit in 256 registers per lane");
  static_assert(BN == 128 || BN == 256, "B swizzle is defined for 16- and 32-chunk rows");
};

// MFMA operand fragments of one K step: A rows (8 K each per lane) and B
// columns (two transposed halves, k 0..3 and 4..7 of the lane's 8).
template <int TM>
struct AFrags {
  bf16x8 a[TM];
};
template <int TN>
struct BFrags {
  i16x4 b[TN][2];
};

// The output tile (partition pr, pc; tile ti, tj inside it) and K range
// (split) of this workgroup: the XCD-aware map, or the native grouped raster
// over the whole tile grid (XCD-oblivious). False when the workgroup has no
// tile. The results depend on blockIdx only; the map's integer divisions run
// on the vector unit, so they are made wave-uniform explicitly: the operand
// descriptors built from them must live in scalar registers.
__device__ __forceinline__ bool tile_of_block_raw(const GemmParams& p, int32_t* pr, int32_t* pc,
                                                  int32_t* ti, int32_t* tj, int32_t* split) {
  *split = 0;
  if (p.remap) return map_tile(p.map, blockIdx.x, pr, pc, ti, tj, split);
  const int32_t TMg = p.map.tiles_m * p.grid_r, TNg = p.map.tiles_n * p.map.grid_c;
  const int32_t t = blockIdx.x;
  if (t >= TMg * TNg) return false;
  const int32_t per_group = p.map.group_m * TNg;
  const int32_t grp = t / per_group, first = grp * p.map.group_m;
  const int32_t gm = min(p.map.group_m, TMg - first);
  const int32_t w = t - grp * per_group;
  const int32_t tig = first + w % gm, tjg = w / gm;
  *pr = tig / p.map.tiles_m;
  *ti = tig - *pr * p.map.tiles_m;
  *pc = tjg / p.map.tiles_n;
  *tj = tjg - *pc * p.map.tiles_n;
  return true;
}

__device__ __forceinline__ bool tile_of_block(const GemmParams& p, int32_t* pr, int32_t* pc,
                                              int32_t* ti, int32_t* tj, int32_t* split) {
  if (!tile_of_block_raw(p, pr, pc, ti, tj, split)) return false;
  *pr = __builtin_amdgcn_readfirstlane(*pr);
  *pc = __builtin_amdgcn_readfirstlane(*pc);
  *ti = __builtin_amdgcn_readfirstlane(*ti);
  *tj = __builtin_amdgcn_readfirstlane(*tj);
  *split = __builtin_amdgcn_readfirstlane(*split);
  return true;
}

// Position of K step k0 in an operand's K blocks: the block offset and the
// element offset inside the block (a block holds kslice elements of K).
// Integer division has no scalar instruction, so the block index is made
// wave-uniform explicitly: the operand descriptors built from it must live
// in scalar registers.
__device__ __forceinline__ void k_start(const OperandAddr& o, int32_t k_elems, int64_t* slice_off,
                                        int32_t* kl) {
  const int32_t kc = __builtin_amdgcn_readfirstlane(k_elems / o.kslice);
  *slice_off = (int64_t)kc * o.slice;
  *kl = __builtin_amdgcn_readfirstlane(k_elems - kc * o.kslice);
}

// Index of tile (pr, pc, ti, tj) among all kernel tiles of C.
__device__ __forceinline__ int64_t tile_id(const GemmParams& p, int32_t pr, int32_t pc, int32_t ti,
                                           int32_t tj) {
  return ((int64_t)(pr * p.map.grid_c + pc) * p.map.tiles_m + ti) * p.map.tiles_n + tj;
}

// Four consecutive C elements at element index idx: alpha * o (+ beta * C),
// stored as bf16 (nearest even) or fp32.
__device__ __forceinline__ void store4(const GemmParams& p, int64_t idx, float* o) {
  const int epi = p.epi;
  const float alpha = p.alpha, beta = p.beta;
  auto scale = [&](const float* old) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      o[j] = epi == 2 ? __builtin_fmaf(alpha, o[j], beta * old[j]) : alpha * o[j];
  };
  if (p.c_f32) {
    float4* dst = reinterpret_cast<float4*>(static_cast<float*>(p.C) + idx);
    if (epi != 0) {
      float old[4] = {0.f, 0.f, 0.f, 0.f};
      if (epi == 2) {
        const float4 c = *dst;
        old[0] = c.x; old[1] = c.y; old[2] = c.z; old[3] = c.w;
      }
      scale(old);
    }
    *dst = make_float4(o[0], o[1], o[2], o[3]);
  } else {
    uint2* dst = reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.C) + idx);
    if (epi != 0) {
      uint2 c = make_uint2(0u, 0u);
      if (epi == 2) c = *dst;
      const float old[4] = {__uint_as_float(c.x << 16), __uint_as_float(c.x & 0xffff0000u),
                            __uint_as_float(c.y << 16), __uint_as_float(c.y & 0xffff0000u)};
      scale(old);
    }
    uint2 v;
    v.x = bf16_rne(o[0]) | (bf16_rne(o[1]) << 16);
    v.y = bf16_rne(o[2]) | (bf16_rne(o[3]) << 16);
    *dst = v;
  }
}

// Where a lane's accumulators sit in C. The product is formed as C^T
// tiles, so with MD x MD MFMA tiles (MD = 16 for bf16, 32 for fp8) lane l
// holds, for each q < Q, C[row][col(q) .. col(q) + 3] of its tile:
//   MD = 16: Q = 1, row = l % 16, col = 4 (l / 16);
//   MD = 32: Q = 4, row = l % 32, col = 8 q + 4 (l / 32).
template <int MD>
struct AccLayout {
  static_assert(MD == 16 || MD == 32, "MFMA tiles are 16x16 or 32x32");
  static constexpr int Q = MD == 16 ? 1 : 4;
  __device__ static __forceinline__ int row(int lane) { return lane & (MD - 1); }
  __device__ static __forceinline__ int col(int lane, int q) {
    return MD == 16 ? 4 * (lane >> 4) : 8 * q + 4 * (lane >> 5);
  }
};

// Position of a lane's four accumulators (group q) in the split-K partial
// tile. The partial is stored in fragment order, so that the 64 lanes of a
// wave write (and the reduce kernel reads) 1 KB contiguous: float4 number
// (((wave * TM + mt) * TN + nt) * Q + q) * 64 + lane, wave = wm * (BN / WN) + wn.
template <int TM, int TN, int Q>
__device__ __forceinline__ int32_t frag_index(int wave, int mt, int nt, int q, int lane) {
  return (((wave * TM + mt) * TN + nt) * Q + q) * 64 + lane;
}

// Epilogue: lane holds C[m][n .. n+3] of each MD x MD MFMA tile (mt, nt) in
// acc[mt][nt][4q .. 4q+3] (AccLayout). Without split-K: C = alpha * acc
// (+ beta * C). With split-K: the fp32 partial tile goes to the workspace at
// tile tile * splits + split, in fragment order, and the reduce kernel
// writes C.
template <int BM, int BN, int MD, int TM, int TN, int WM, int WN, typename Acc>
__device__ __forceinline__ void store_tile(const GemmParams& p, const Acc (&acc)[TM][TN],
                                           int32_t pr, int32_t pc, int32_t ti, int32_t tj,
                                           int32_t split, int wm, int wn, int lane) {
  using L = AccLayout<MD>;
  const int64_t c_tile = pr * p.c.part + pc * p.c.slice + (int64_t)(ti * BM) * p.c.ld + tj * BN;
  float* part = p.ws ? p.ws + (tile_id(p, pr, pc, ti, tj) * p.map.splits + split) * (BM * BN) : nullptr;
  const int wave = wm * (BN / WN) + wn;
#pragma unroll
  for (int mt = 0; mt < TM; ++mt) {
    const int m = wm * WM + mt * MD + L::row(lane);
#pragma unroll
    for (int nt = 0; nt < TN; ++nt) {
#pragma unroll
      for (int q = 0; q < L::Q; ++q) {
        const int n = wn * WN + nt * MD + L::col(lane, q);
        float o[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) o[j] = acc[mt][nt][4 * q + j];
        if (part)
          reinterpret_cast<float4*>(part)[frag_index<TM, TN, L::Q>(wave, mt, nt, q, lane)] =
              make_float4(o[0], o[1], o[2], o[3]);
        else
          store4(p, c_tile + (int64_t)m * p.c.ld + n, o);
      }
    }
  }
}

// Epilogue of the kernels with 16x16 MFMA tiles (bf16, fp8 16x16x128) for a
// plain bf16 C (alpha 1, beta 0, no split-K), staged through LDS so that C leaves the CU in whole 128-byte
// lines. The direct form (store_tile) writes 8 bytes per lane, i.e. 32-byte
// pieces of 16 rows per instruction, and a CU then issues its C tile at
// about 17 GB/s. Here each wave first writes its bf16 values into the
// (then idle) stage buffers: rows 0 .. BM/2 - 1 of the tile into `lo`,
// rows BM/2 .. BM - 1 into `hi`, row pitch BN * 2 bytes, with the 16-byte
// chunk index XORed with (row mod 16) so that the 16 rows of one write fall
// in distinct banks. Then every wave copies BM / NW whole rows to C, 16
// bytes per lane. NT marks the stores to C non-temporal (C is not read back
// by the kernel); the 64-K-stage kernel uses it, where its Qwen3-shaped
// launches (gate/up, dH) ran 1.5-3 % faster with it, measured alternating,
// and so does the pipelined fp8 kernel.
template <int BM, int BN, int NW, int TM, int TN, int WM, int WN, bool NT = false>
__device__ __forceinline__ void store_tile_staged(const GemmParams& p, const f32x4 (&acc)[TM][TN],
                                                  char* lo, char* hi, int32_t pr, int32_t pc,
                                                  int32_t ti, int32_t tj, int wm, int wn, int wave,
                                                  int lane) {
  constexpr int ROWB = BN * 2;              // bytes per C row in LDS and in C
  constexpr int CPR = BN / 8;               // 16-byte chunks per row
  constexpr int HALF = BM / 2;              // rows per half
  constexpr int RPI = 64 / CPR;             // rows per wave-wide 16-byte access
  constexpr int RPW = BM / NW;              // rows copied out per wave
  static_assert(WM == HALF, "a wave's rows lie in one half");
  static_assert(RPW % RPI == 0, "whole accesses per wave");
  // No wave reads the stage buffers any more and no load into them is in
  // flight (the direct-to-LDS loads of the last steps included).
  __builtin_amdgcn_s_waitcnt(0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  char* half = wm ? hi : lo;
#pragma unroll
  for (int mt = 0; mt < TM; ++mt) {
    const int r = mt * 16 + (lane & 15);
#pragma unroll
    for (int nt = 0; nt < TN; ++nt) {
      const int col = wn * WN + nt * 16 + 4 * (lane >> 4);
      uint2 v;
      v.x = bf16_rne(acc[mt][nt][0]) | (bf16_rne(acc[mt][nt][1]) << 16);
      v.y = bf16_rne(acc[mt][nt][2]) | (bf16_rne(acc[mt][nt][3]) << 16);
      *reinterpret_cast<uint2*>(half + r * ROWB + (((col >> 3) ^ (r & 15)) << 4) + ((col >> 2) & 1) * 8) = v;
    }
  }
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(63, 0));
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  uint16_t* C = static_cast<uint16_t*>(p.C) + pr * p.c.part + pc * p.c.slice +
                (int64_t)(ti * BM) * p.c.ld + tj * BN;
  const int c = lane % CPR;
#pragma unroll
  for (int i = 0; i < RPW / RPI; ++i) {
    const int row = wave * RPW + i * RPI + lane / CPR;
    const int r = row % HALF;
    const uint4 v = *reinterpret_cast<const uint4*>((row < HALF ? lo : hi) + r * ROWB + ((c ^ (r & 15)) << 4));
    uint4* dst = reinterpret_cast<uint4*>(C + (int64_t)row * p.c.ld + c * 8);
    if constexpr (NT)
      __builtin_nontemporal_store(__builtin_bit_cast(i32x4, v), reinterpret_cast<i32x4*>(dst));
    else
      *dst = v;
  }
}

// Split-K reduction. Each tile is cut into kChunks chunks of 256 float4
// (fragment order); workgroup w handles chunk (w >> 3) % kChunks of the tile
// that workgroup ((w >> 3) / kChunks) * 8 + (w & 7) of the unsplit GEMM
// computes, so it runs on the XCD that wrote the partials. Each thread sums
// its float4 over the splits in ascending order and writes C through store4.
// MD is the MFMA tile of the GEMM kernel that wrote the partials.
template <int BM, int BN, int WGN, int MD>
__global__ void __launch_bounds__(256) splitk_reduce_kernel(GemmParams p) {
  using L = AccLayout<MD>;
  constexpr int WM = BM / 2, WN = BN / WGN;
  constexpr int TM = WM / MD, TN = WN / MD;
  constexpr int kChunks = BM * BN / (4 * 256);
  const int64_t slot = blockIdx.x >> 3;
  const int32_t chunk = (int32_t)(slot % kChunks);
  int32_t pr, pc, ti, tj, split;
  if (!map_tile(p.map, ((slot / kChunks) << 3) | (blockIdx.x & 7), &pr, &pc, &ti, &tj, &split))
    return;
  const int32_t f = chunk * 256 + threadIdx.x;
  const int lane = f & 63;
  int r = f >> 6;
  const int q = r % L::Q;
  r /= L::Q;
  const int nt = r % TN;
  r /= TN;
  const int mt = r % TM;
  const int wave = r / TM;
  const int wm = wave / (BN / WN), wn = wave % (BN / WN);
  const int m = wm * WM + mt * MD + L::row(lane);
  const int n = wn * WN + nt * MD + L::col(lane, q);
  const int32_t S = p.splits_total;
  const float4* part = reinterpret_cast<const float4*>(p.ws + tile_id(p, pr, pc, ti, tj) * S * (BM * BN)) + f;
  float o[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int s = 0; s < S; ++s) {
    const float4 v = part[(int64_t)s * (BM * BN / 4)];
    o[0] += v.x; o[1] += v.y; o[2] += v.z; o[3] += v.w;
  }
  const int64_t c_tile = pr * p.c.part + pc * p.c.slice + (int64_t)(ti * BM) * p.c.ld + tj * BN;
  store4(p, c_tile + (int64_t)m * p.c.ld + n, o);
}

// Writes one wave's phase timeline once its C stores have been issued (not
// waited for, as in the ordinary launch): words 0-3 real-time counter
// (start, after prologue, after K loop, after the stores' issue), 4-5
// shader clock (start, after K loop), 6 the XCD id, 7 the raw HW_ID
// register (its CU, SH and SE fields name the CU). Lane 0 writes.
__device__ __forceinline__ void record_timeline(uint64_t* o, const uint64_t (&rt)[3],
                                                const uint64_t (&clk)[2], int lane) {
  const uint64_t t_end = __builtin_amdgcn_s_memrealtime();
  uint32_t xcc, hw;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(hw));
  if (lane == 0) {
    o[0] = rt[0]; o[1] = rt[1]; o[2] = rt[2]; o[3] = t_end;
    o[4] = clk[0]; o[5] = clk[1]; o[6] = xcc; o[7] = hw;
  }
}

template <int BM, int BN, int WGN>
__global__ void __launch_bounds__(128 * WGN, WGN / 2) gemm_kernel(GemmParams p) {
  // The host pass only needs the launch stub; the body uses device-only
  // buffer-resource builtins.
#if defined(__HIP_DEVICE_COMPILE__)
  using T = Tile<BM, BN, WGN>;
  constexpr int NS = kStagesBf16;
  __shared__ __attribute__((aligned(1024))) char smA[NS][T::A_BYTES];
  __shared__ __attribute__((aligned(1024))) char smB[NS][T::B_BYTES];

  // Phase timeline (debug launches only; the branch is uniform): the
  // 100 MHz real-time counter at the start, after the prologue, after the
  // K loop and after the epilogue's stores, and the shader clock counter at
  // the start and after the K loop.
  const bool tl_on = p.timeline != nullptr;
  uint64_t tl_rt[3] = {0, 0, 0}, tl_clk[2] = {0, 0};
  if (tl_on) {
    tl_rt[0] = __builtin_amdgcn_s_memrealtime();
    tl_clk[0] = __builtin_amdgcn_s_memtime();
  }
  int32_t pr, pc, ti, tj, split;
  if (!tile_of_block(p, &pr, &pc, &ti, &tj, &split)) return;
  // K range of this workgroup: steps [k0, k0 + ksteps) (all of K without split-K)
  const int32_t k0 = __builtin_amdgcn_readfirstlane(split * p.ksteps_per_split);
  const int32_t ksteps = __builtin_amdgcn_readfirstlane(min(p.ksteps, k0 + p.ksteps_per_split) - k0);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;

  // ---- global -> LDS: per-lane byte offsets from the K step's tile corner ----
  // A load i of this wave fills LDS rows 16*(wave*NA+i) .. +15 (64 B each).
  uint32_t a_voff[T::NA];
#pragma unroll
  for (int i = 0; i < T::NA; ++i) {
    const int row = 16 * (wave * T::NA + i) + (lane >> 2);
    const int chunk = (lane & 3) ^ swz_a16(row);
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
  // A fragment of MFMA tile mt: lane l reads row wm*WM + 16 mt + l % 16,
  // K chunk l / 16 (8 bf16). B fragment of tile nt, half r: lane l = 16 g + s
  // reads 4 columns of row 8 g + 4 r + s / 4 for the transposed read.
  int32_t a_rd;
  {
    const int row = wm * T::WM + (lane & 15);
    a_rd = row * 64 + (((lane >> 4) ^ swz_a16(row)) * 16);
  }
  int32_t b_rd[T::TN][2];
  {
    const int g = lane >> 4, s = lane & 15;
#pragma unroll
    for (int nt = 0; nt < T::TN; ++nt) {
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int krow = 8 * g + 4 * r + (s >> 2);
        const int col = wn * T::WN + nt * 16 + 4 * (s & 3);
        b_rd[nt][r] = krow * (BN * 2) + (((col >> 3) ^ swz_b(krow)) * 16) + ((col >> 2) & 1) * 8;
      }
    }
  }

  // ---- operand corners; K-slice block advances every kslice columns/rows ----
  const uint16_t* a_base = p.A + pr * p.a.part + (int64_t)(ti * BM) * p.a.ld;
  const uint16_t* b_base = p.B + pc * p.b.part + tj * BN;
  int64_t a_slice_off, b_slice_off;
  int32_t a_kl, b_kl;
  k_start(p.a, k0 * kBK, &a_slice_off, &a_kl);
  k_start(p.b, k0 * kBK, &b_slice_off, &b_kl);
  // Byte address of the next K step's A and B corners. It advances by one
  // step at a time; after the last step of a CCL K block it jumps to the
  // start of the next block.
  const char* a_next = reinterpret_cast<const char*>(a_base + a_slice_off + a_kl);
  const char* b_next = reinterpret_cast<const char*>(b_base + b_slice_off + (int64_t)b_kl * p.b.ld);
  const int32_t a_steps = p.a.kslice / kBK, b_steps = p.b.kslice / kBK;   // steps per block
  int32_t a_left = a_steps - a_kl / kBK, b_left = b_steps - b_kl / kBK;   // left in this block
  const int64_t a_adv = kBK * 2, b_adv = (int64_t)kBK * p.b.ld * 2;
  const int64_t a_jump = (p.a.slice - p.a.kslice) * 2;
  const int64_t b_jump = (p.b.slice - (int64_t)p.b.kslice * p.b.ld) * 2;

  // Descriptors of the next K step to be loaded. With live == false they
  // cover zero bytes: every load is out of range, touches no memory and
  // writes zeros to the (unused) stage.
  struct StageSrc {
    i32x4 ra, rb;
  };
  auto next_src = [&](bool live) {
    StageSrc d;
    d.ra = buffer_rsrc(a_next, live ? a_extent : 0);
    d.rb = buffer_rsrc(b_next, live ? b_extent : 0);
    // advance to the next K step (branch-free; past the last step the
    // corners are only used with empty descriptors)
    const bool a_wrap = --a_left == 0;
    a_next += a_adv + (a_wrap ? a_jump : 0);
    a_left = a_wrap ? a_steps : a_left;
    const bool b_wrap = --b_left == 0;
    b_next += b_adv + (b_wrap ? b_jump : 0);
    b_left = b_wrap ? b_steps : b_left;
    return d;
  };
  // Descriptors of four consecutive K steps at once (the rounds path): the
  // steps of a round address their K slice through the loads' scalar
  // offsets (so_a[j], so_b[j]); the corners advance by four steps. Only
  // used where no round straddles a CCL K block (a_left is then a multiple
  // of 4 here, or the operand has a single block).
  const int32_t a_extent4 = (BM - 1) * p.a.ld * 2 + 4 * kBK * 2;
  const int32_t b_extent4 = (4 * kBK - 1) * p.b.ld * 2 + BN * 2;
  const uint32_t so_a[4] = {0u, (uint32_t)a_adv, (uint32_t)(2 * a_adv), (uint32_t)(3 * a_adv)};
  const uint32_t so_b[4] = {0u, (uint32_t)b_adv, (uint32_t)(2 * b_adv), (uint32_t)(3 * b_adv)};
  auto round_src = [&]() {
    StageSrc d;
    d.ra = buffer_rsrc(a_next, a_extent4);
    d.rb = buffer_rsrc(b_next, b_extent4);
    const bool a_wrap = a_left == 4;
    a_next += 4 * a_adv + (a_wrap ? a_jump : 0);
    a_left = a_wrap ? a_steps : a_left - 4;
    const bool b_wrap = b_left == 4;
    b_next += 4 * b_adv + (b_wrap ? b_jump : 0);
    b_left = b_wrap ? b_steps : b_left - 4;
    return d;
  };
  // Load i (0 .. NL-1) of this wave for one stage; j >= 0 selects the
  // scalar offsets of step j of a round.
  auto load_one = [&](const StageSrc& d, int j, char* smA, char* smB, int i) {
    if (i < T::NA) {
      char* dst = smA + (wave * T::NA + i) * 1024;
      if (j < 0) lds_dma16(d.ra, a_voff[i], dst);
      else lds_dma16_so(d.ra, a_voff[i], so_a[j], dst);
    } else {
      char* dst = smB + (wave * T::NB + (i - T::NA)) * 1024;
      if (j < 0) lds_dma16(d.rb, b_voff[i - T::NA], dst);
      else lds_dma16_so(d.rb, b_voff[i - T::NA], so_b[j], dst);
    }
  };
  auto load_stage = [&](char* smA, char* smB, bool live) {
    const StageSrc d = next_src(live);
#pragma unroll
    for (int i = 0; i < T::NL; ++i) load_one(d, -1, smA, smB, i);
  };

  constexpr int kHalfM = T::TM / 2;               // A fragments per half step
  AFrags<T::TM> fa;
  BFrags<T::TN> fb0, fb1;
  auto read_a = [&](const char* smA, int mt) {
    fa.a[mt] = *(const lds_bf16x8*)(smA + a_rd + mt * 16 * 64);
  };
  // B read i (0 .. 2 TN - 1): tile i / 2, half i % 2.
  auto read_b = [&](const char* smB, BFrags<T::TN>& fb, int i) {
    const int nt = i >> 1, r = i & 1;
    fb.b[nt][r] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(smB + b_rd[nt][r]));
  };

  f32x4 acc[T::TM][T::TN];
#pragma unroll
  for (int i = 0; i < T::TM; ++i)
#pragma unroll
    for (int j = 0; j < T::TN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[i][j][v] = 0.f;

  auto mfma_one = [&](const BFrags<T::TN>& fb, int mt, int nt) {
    const bf16x8 bv = __builtin_bit_cast(
        bf16x8, __builtin_shufflevector(fb.b[nt][0], fb.b[nt][1], 0, 1, 2, 3, 4, 5, 6, 7));
    acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bv, fa.a[mt], acc[mt][nt], 0, 0, 0);
  };

  // Wait for the own loads of the next stage (the later stages' loads stay
  // in flight) and for this wave's LDS reads, then for every wave: after
  // this barrier the next stage is complete in LDS, and nobody reads the
  // stage that the next load reuses. An LDS-only wait: a full fence would
  // also wait for the in-flight direct-to-LDS loads of the later stages.
  auto stage_barrier = [&]() {
    __builtin_amdgcn_s_waitcnt(waitcnt_imm((NS - 2) * T::NL, 0));
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  // One K step on stage (smA, smB). On entry A fragments 0 .. kHalfM-1 and
  // the B fragments fb hold this stage's data. First half: the MFMAs of A
  // fragments 0 .. kHalfM-1, each followed by at most one memory
  // instruction: the reads of A fragments kHalfM .. TM-1 of this stage, then
  // the direct-to-LDS loads of the step NS-1 ahead into (lA, lB). After
  // the stage barrier, the second half runs the MFMAs of A fragments
  // kHalfM .. TM-1 and reads the next stage (nA, nB): A fragments
  // 0 .. kHalfM-1 (no longer needed) and all B fragments into fbn. The order
  // is pinned so the matrix pipe always has the next MFMA ready while the
  // memory instructions drain behind it.
  auto step = [&](const char* smA, const char* smB, const BFrags<T::TN>& fb, BFrags<T::TN>& fbn,
                  char* lA, char* lB, const char* nA, const char* nB, const StageSrc& d, int j) {
    constexpr int kMfmaHalf = kHalfM * T::TN;
    constexpr int kOps1 = kHalfM + T::NL;
#pragma unroll
    for (int i = 0; i < kMfmaHalf; ++i) {
      mfma_one(fb, i / T::TN, i % T::TN);
      if (i < kHalfM) read_a(smA, kHalfM + i);
      else if (i < kOps1) load_one(d, j, lA, lB, i - kHalfM);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = kMfmaHalf; i < kOps1; ++i) {
      if (i < kHalfM) read_a(smA, kHalfM + i);
      else load_one(d, j, lA, lB, i - kHalfM);
    }
    __builtin_amdgcn_sched_barrier(0);
    stage_barrier();
    constexpr int kOps2 = kHalfM + 2 * T::TN;
#pragma unroll
    for (int i = 0; i < kMfmaHalf; ++i) {
      mfma_one(fb, kHalfM + i / T::TN, i % T::TN);
      if (i < kHalfM) read_a(nA, i);
      else if (i < kOps2) read_b(nB, fbn, i - kHalfM);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = kMfmaHalf; i < kOps2; ++i) {
      if (i < kHalfM) read_a(nA, i);
      else read_b(nB, fbn, i - kHalfM);
    }
    __builtin_amdgcn_sched_barrier(0);
  };

  // Prologue: the first NS-1 stages in flight, then stage 0's first fragments.
#pragma unroll
  for (int j = 0; j < NS - 1; ++j) load_stage(smA[j], smB[j], j < ksteps);
  stage_barrier();
  if (tl_on) tl_rt[1] = __builtin_amdgcn_s_memrealtime();
#pragma unroll
  for (int mt = 0; mt < kHalfM; ++mt) read_a(smA[0], mt);
#pragma unroll
  for (int i = 0; i < 2 * T::TN; ++i) read_b(smB[0], fb0, i);
  // Step s works on stage s % NS, loads stage (s + NS - 1) % NS (the step
  // NS-1 ahead) and reads stage (s + 1) % NS; the B fragment sets alternate.
  // ph is s modulo a multiple of NS and of 2, known at compile time.
  auto phase_step = [&](int ph, const StageSrc& d, int j) {
    step(smA[ph % NS], smB[ph % NS], ph % 2 ? fb1 : fb0, ph % 2 ? fb0 : fb1,
         smA[(ph + NS - 1) % NS], smB[(ph + NS - 1) % NS], smA[(ph + 1) % NS],
         smB[(ph + 1) % NS], d, j);
  };
  // One step with its own descriptors (live: the step it loads exists).
  auto single_step = [&](int ph, int32_t s) {
    const StageSrc d = next_src(s + NS - 1 < ksteps);
    phase_step(ph, d, -1);
  };
  constexpr int kRound = NS % 2 ? 2 * NS : NS;
  int32_t s = 0;
  if (NS == 4 && p.round_fast) {
    // Rounds path. Step 0 alone; then rounds of 4 steps (s = 1 mod 4) whose
    // loads (steps s+3 .. s+6, a 4-aligned group) are all live and share
    // one pair of descriptors; the remaining steps (at most 6) alone. Whole
    // rounds run branch-free, so the compiler tracks the outstanding LDS
    // reads exactly and waits only for the fragments each MFMA needs.
    single_step(0, 0);
    for (s = 1; s + 7 <= ksteps; s += 4) {
      const StageSrc d = round_src();
#pragma unroll
      for (int j = 0; j < 4; ++j) phase_step(1 + j, d, j);
    }
#pragma unroll
    for (int t = 0; t < 6; ++t)
      if (s + t < ksteps) single_step(1 + t, s + t);
  } else {
    // Per-step path: whole rounds of kRound steps branch-free, then the
    // last, partial round under conditions.
    const int32_t full = ksteps - ksteps % kRound;
    for (; s < full; s += kRound) {
#pragma unroll
      for (int j = 0; j < kRound; ++j) single_step(j, s + j);
    }
#pragma unroll
    for (int j = 0; j < kRound - 1; ++j)
      if (s + j < ksteps) single_step(j, s + j);
  }

  if (tl_on) {
    tl_rt[2] = __builtin_amdgcn_s_memrealtime();
    tl_clk[1] = __builtin_amdgcn_s_memtime();
  }
  static_assert((BM / 2) * BN * 2 <= NS * T::A_BYTES && (BM / 2) * BN * 2 <= NS * T::B_BYTES,
                "each half of the bf16 C tile fits in one operand's stage buffers");
  if (p.epi == 0 && !p.c_f32 && !p.ws)
    store_tile_staged<BM, BN, T::NW, T::TM, T::TN, T::WM, T::WN>(p, acc, &smA[0][0], &smB[0][0], pr,
                                                                 pc, ti, tj, wm, wn, wave, lane);
  else
    store_tile<BM, BN, 16, T::TM, T::TN, T::WM, T::WN>(p, acc, pr, pc, ti, tj, split, wm, wn, lane);
  if (tl_on) record_timeline(p.timeline + ((int64_t)blockIdx.x * T::NW + wave) * kTimelineWords,
                             tl_rt, tl_clk, lane);
#endif
}

// ---------------------------------------------------------------------------
// bf16 with 64-K stages, for the output tiles below 256x256 (8 waves). A
// stage holds 64 K, so each A row in LDS is 128 bytes: the
// direct-to-LDS loads fetch whole 128-byte lines of A, which a CU streams
// from L2 about 1.5x faster than the half lines of 32-K stages when most
// CUs load at once. Each step runs the MFMAs of two 32-K sub-steps (kk = 0,
// 1) around one barrier:
//  * first half: the MFMAs of sub-step 0 (fragments fa0/fb0), behind them
//    the reads of sub-step 1's fragments (fa1/fb1) and the direct-to-LDS
//    loads of the stage NS-1 steps ahead;
//  * stage barrier;
//  * second half: the MFMAs of sub-step 1, behind them the reads of the next
//    stage's sub-step 0 fragments into fa0/fb0.
// A rows: chunk c (16 bytes) of row r sits at chunk c ^ swz_a64(r); the 16
// rows x 4 chunks of one A fragment read then fall in distinct bank slots
// (checked against the measured ds_read_b128 grouping: lanes with equal
// parity of lane bits 2..4 are served together). B rows are as in the 32-K
// kernel, twice as many per stage.
// ---------------------------------------------------------------------------

constexpr int kBK64 = 64;        // K extent of one stage of gemm_k64_kernel

__device__ __forceinline__ int swz_a64(int row) { return (row >> 1) & 7; }

template <int BM, int BN>
struct Tile64 {
  static constexpr int WGN = 4;
  static constexpr int NW = 8;                         // waves per workgroup
  static constexpr int THREADS = 64 * NW;
  static constexpr int WM = BM / 2, WN = BN / WGN;     // wave tile
  static constexpr int TM = WM / 16, TN = WN / 16;     // MFMA tiles per wave
  static constexpr int A_BYTES = BM * kBK64 * 2;       // one stage
  static constexpr int B_BYTES = kBK64 * BN * 2;
  static constexpr int NA = A_BYTES / (1024 * NW);     // A loads per wave per stage (8 rows each)
  static constexpr int CPR_B = BN / 8;                 // 16-byte chunks per B row
  static constexpr int RPI_B = 64 / CPR_B;             // B rows per load instruction
  static constexpr int NB = B_BYTES / (1024 * NW);     // B loads per wave per stage
  static constexpr int NL = NA + NB;
  // as many stages as 160 KiB holds, at most 4: 3 for 256x128 and
  // 128x256, 4 for 128x128
  static constexpr int NS = (160 * 1024) / (A_BYTES + B_BYTES) >= 4 ? 4 : 3;
  static_assert(BM * BN < 256 * 256, "256x256 tiles use the 32-K stages");
  static_assert(NA >= 1 && NB >= 1 && TN >= 1 && TM >= 1, "tile too small for the wave grid");
  static_assert(NS * (A_BYTES + B_BYTES) <= 160 * 1024, "LDS stages exceed 160 KiB");
  static_assert((NS - 2) * NL <= 63, "the stage wait count exceeds vmcnt's range");
  static_assert(BN == 128 || BN == 256, "B swizzle is defined for 16- and 32-chunk rows");
};

template <int BM, int BN>
__global__ void __launch_bounds__(512, 2) gemm_k64_kernel(GemmParams p) {
#if defined(__HIP_DEVICE_COMPILE__)
  using T = Tile64<BM, BN>;
  constexpr int NS = T::NS;
  __shared__ __attribute__((aligned(1024))) char smA[NS][T::A_BYTES];
  __shared__ __attribute__((aligned(1024))) char smB[NS][T::B_BYTES];

  const bool tl_on = p.timeline != nullptr;
  uint64_t tl_rt[3] = {0, 0, 0}, tl_clk[2] = {0, 0};
  if (tl_on) {
    tl_rt[0] = __builtin_amdgcn_s_memrealtime();
    tl_clk[0] = __builtin_amdgcn_s_memtime();
  }
  int32_t pr, pc, ti, tj, split;
  if (!tile_of_block(p, &pr, &pc, &ti, &tj, &split)) return;
  // K range of this workgroup: steps [k0, k0 + ksteps) (all of K without split-K)
  const int32_t k0 = __builtin_amdgcn_readfirstlane(split * p.ksteps_per_split);
  const int32_t ksteps = __builtin_amdgcn_readfirstlane(min(p.ksteps, k0 + p.ksteps_per_split) - k0);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / T::WGN, wn = wave % T::WGN;

  // ---- global -> LDS: per-lane byte offsets from the K step's tile corner ----
  // A load i of this wave fills LDS rows 8*(wave*NA+i) .. +7 (128 B each);
  // the lane at LDS chunk q of its row fetches global chunk q ^ swz_a64(row).
  uint32_t a_voff[T::NA];
#pragma unroll
  for (int i = 0; i < T::NA; ++i) {
    const int row = 8 * (wave * T::NA + i) + (lane >> 3);
    const int chunk = (lane & 7) ^ swz_a64(row);
    a_voff[i] = (uint32_t)(row * p.a.ld + chunk * 8) * 2u;
  }
  uint32_t b_voff[T::NB];
#pragma unroll
  for (int i = 0; i < T::NB; ++i) {
    const int row = T::RPI_B * (wave * T::NB + i) + lane / T::CPR_B;
    const int chunk = (lane % T::CPR_B) ^ swz_b(row);
    b_voff[i] = (uint32_t)(row * p.b.ld + chunk * 8) * 2u;
  }
  const int32_t a_extent = (BM - 1) * p.a.ld * 2 + kBK64 * 2;
  const int32_t b_extent = (kBK64 - 1) * p.b.ld * 2 + BN * 2;

  // ---- LDS fragment read offsets (bytes), sub-step kk ----
  // A fragment of MFMA tile mt: lane l reads row wm*WM + 16 mt + l % 16,
  // K chunk 4 kk + l / 16; the swizzle depends on the row only through
  // (row >> 1) & 7, the same for every mt.
  int32_t a_rd[2];
  {
    const int row = wm * T::WM + (lane & 15);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
      a_rd[kk] = row * 128 + (((4 * kk + (lane >> 4)) ^ swz_a64(row)) * 16);
  }
  int32_t b_rd[T::TN][2];
  {
    const int g = lane >> 4, s = lane & 15;
#pragma unroll
    for (int nt = 0; nt < T::TN; ++nt) {
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int krow = 8 * g + 4 * r + (s >> 2);
        const int col = wn * T::WN + nt * 16 + 4 * (s & 3);
        b_rd[nt][r] = krow * (BN * 2) + (((col >> 3) ^ swz_b(krow)) * 16) + ((col >> 2) & 1) * 8;
      }
    }
  }
  constexpr int kB_KK = 32 * BN * 2;            // bytes between the two sub-steps' B rows

  // ---- operand corners; K-slice block advances every kslice columns/rows ----
  const uint16_t* a_base = p.A + pr * p.a.part + (int64_t)(ti * BM) * p.a.ld;
  const uint16_t* b_base = p.B + pc * p.b.part + tj * BN;
  int64_t a_slice_off, b_slice_off;
  int32_t a_kl, b_kl;
  k_start(p.a, k0 * kBK64, &a_slice_off, &a_kl);
  k_start(p.b, k0 * kBK64, &b_slice_off, &b_kl);
  const char* a_next = reinterpret_cast<const char*>(a_base + a_slice_off + a_kl);
  const char* b_next = reinterpret_cast<const char*>(b_base + b_slice_off + (int64_t)b_kl * p.b.ld);
  const int32_t a_steps = p.a.kslice / kBK64, b_steps = p.b.kslice / kBK64;
  int32_t a_left = a_steps - a_kl / kBK64, b_left = b_steps - b_kl / kBK64;
  const int64_t a_adv = kBK64 * 2, b_adv = (int64_t)kBK64 * p.b.ld * 2;
  const int64_t a_jump = (p.a.slice - p.a.kslice) * 2;
  const int64_t b_jump = (p.b.slice - (int64_t)p.b.kslice * p.b.ld) * 2;

  struct StageSrc {
    i32x4 ra, rb;
  };
  auto next_src = [&](bool live) {
    StageSrc d;
    d.ra = buffer_rsrc(a_next, live ? a_extent : 0);
    d.rb = buffer_rsrc(b_next, live ? b_extent : 0);
    const bool a_wrap = --a_left == 0;
    a_next += a_adv + (a_wrap ? a_jump : 0);
    a_left = a_wrap ? a_steps : a_left;
    const bool b_wrap = --b_left == 0;
    b_next += b_adv + (b_wrap ? b_jump : 0);
    b_left = b_wrap ? b_steps : b_left;
    return d;
  };
  const int32_t a_extent4 = (BM - 1) * p.a.ld * 2 + 4 * kBK64 * 2;
  const int32_t b_extent4 = (4 * kBK64 - 1) * p.b.ld * 2 + BN * 2;
  const uint32_t so_a[4] = {0u, (uint32_t)a_adv, (uint32_t)(2 * a_adv), (uint32_t)(3 * a_adv)};
  const uint32_t so_b[4] = {0u, (uint32_t)b_adv, (uint32_t)(2 * b_adv), (uint32_t)(3 * b_adv)};
  auto round_src = [&]() {
    StageSrc d;
    d.ra = buffer_rsrc(a_next, a_extent4);
    d.rb = buffer_rsrc(b_next, b_extent4);
    const bool a_wrap = a_left == 4;
    a_next += 4 * a_adv + (a_wrap ? a_jump : 0);
    a_left = a_wrap ? a_steps : a_left - 4;
    const bool b_wrap = b_left == 4;
    b_next += 4 * b_adv + (b_wrap ? b_jump : 0);
    b_left = b_wrap ? b_steps : b_left - 4;
    return d;
  };
  auto load_one = [&](const StageSrc& d, int j, char* sA, char* sB, int i) {
    if (i < T::NA) {
      char* dst = sA + (wave * T::NA + i) * 1024;
      if (j < 0) lds_dma16(d.ra, a_voff[i], dst);
      else lds_dma16_so(d.ra, a_voff[i], so_a[j], dst);
    } else {
      char* dst = sB + (wave * T::NB + (i - T::NA)) * 1024;
      if (j < 0) lds_dma16(d.rb, b_voff[i - T::NA], dst);
      else lds_dma16_so(d.rb, b_voff[i - T::NA], so_b[j], dst);
    }
  };
  auto load_stage = [&](char* sA, char* sB, bool live) {
    const StageSrc d = next_src(live);
#pragma unroll
    for (int i = 0; i < T::NL; ++i) load_one(d, -1, sA, sB, i);
  };

  AFrags<T::TM> fa0, fa1;
  BFrags<T::TN> fb0, fb1;
  auto read_a = [&](const char* sA, AFrags<T::TM>& fa, int kk, int mt) {
    fa.a[mt] = *(const lds_bf16x8*)(sA + a_rd[kk] + mt * 16 * 128);
  };
  auto read_b = [&](const char* sB, BFrags<T::TN>& fb, int kk, int i) {
    const int nt = i >> 1, r = i & 1;
    fb.b[nt][r] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(sB + b_rd[nt][r] + kk * kB_KK));
  };

  f32x4 acc[T::TM][T::TN];
#pragma unroll
  for (int i = 0; i < T::TM; ++i)
#pragma unroll
    for (int j = 0; j < T::TN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[i][j][v] = 0.f;

  auto mfma_one = [&](const AFrags<T::TM>& fa, const BFrags<T::TN>& fb, int mt, int nt) {
    const bf16x8 bv = __builtin_bit_cast(
        bf16x8, __builtin_shufflevector(fb.b[nt][0], fb.b[nt][1], 0, 1, 2, 3, 4, 5, 6, 7));
    acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bv, fa.a[mt], acc[mt][nt], 0, 0, 0);
  };
  auto stage_barrier = [&]() {
    __builtin_amdgcn_s_waitcnt(waitcnt_imm((NS - 2) * T::NL, 0));
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  // One step on stage (sA, sB); on entry fa0/fb0 hold its sub-step 0.
  auto step = [&](const char* sA, const char* sB, char* lA, char* lB, const char* nA,
                  const char* nB, const StageSrc& d, int j) {
    constexpr int kMfma = T::TM * T::TN;
    constexpr int kReads = T::TM + 2 * T::TN;
    constexpr int kOps1 = kReads + T::NL;
#pragma unroll
    for (int i = 0; i < kMfma; ++i) {
      mfma_one(fa0, fb0, i / T::TN, i % T::TN);
      if (i < T::TM) read_a(sA, fa1, 1, i);
      else if (i < kReads) read_b(sB, fb1, 1, i - T::TM);
      else if (i < kOps1) load_one(d, j, lA, lB, i - kReads);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = kMfma; i < kOps1; ++i) {
      if (i < T::TM) read_a(sA, fa1, 1, i);
      else if (i < kReads) read_b(sB, fb1, 1, i - T::TM);
      else load_one(d, j, lA, lB, i - kReads);
    }
    __builtin_amdgcn_sched_barrier(0);
    stage_barrier();
#pragma unroll
    for (int i = 0; i < kMfma; ++i) {
      mfma_one(fa1, fb1, i / T::TN, i % T::TN);
      if (i < T::TM) read_a(nA, fa0, 0, i);
      else if (i < kReads) read_b(nB, fb0, 0, i - T::TM);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = kMfma; i < kReads; ++i) {
      if (i < T::TM) read_a(nA, fa0, 0, i);
      else read_b(nB, fb0, 0, i - T::TM);
    }
    __builtin_amdgcn_sched_barrier(0);
  };

  // Prologue: the first NS-1 stages in flight, then stage 0's sub-step 0.
#pragma unroll
  for (int j = 0; j < NS - 1; ++j) load_stage(smA[j], smB[j], j < ksteps);
  stage_barrier();
  if (tl_on) tl_rt[1] = __builtin_amdgcn_s_memrealtime();
#pragma unroll
  for (int mt = 0; mt < T::TM; ++mt) read_a(smA[0], fa0, 0, mt);
#pragma unroll
  for (int i = 0; i < 2 * T::TN; ++i) read_b(smB[0], fb0, 0, i);
  // Step s works on stage s % NS, loads stage (s + NS - 1) % NS and reads
  // stage (s + 1) % NS; ph is s modulo a multiple of NS.
  auto phase_step = [&](int ph, const StageSrc& d, int j) {
    step(smA[ph % NS], smB[ph % NS], smA[(ph + NS - 1) % NS], smB[(ph + NS - 1) % NS],
         smA[(ph + 1) % NS], smB[(ph + 1) % NS], d, j);
  };
  auto single_step = [&](int ph, int32_t s) {
    const StageSrc d = next_src(s + NS - 1 < ksteps);
    phase_step(ph, d, -1);
  };
  int32_t s = 0;
  if (p.round_fast) {
    // Rounds of 4 steps whose loads (steps s+NS-1 .. s+NS+2) form a
    // 4-aligned group, all live, sharing one pair of descriptors. The first
    // kFirst steps run alone so that the first round's loads start
    // 4-aligned; a loop iteration runs kLoop steps (a multiple of NS and of
    // 4, so every phase is known at compile time); the remaining steps
    // (fewer than kLoop + NS - 1) run alone.
    constexpr int kFirst = (4 - (NS - 1) % 4) % 4;
    constexpr int kLoop = NS % 4 == 0 ? NS : 4 * NS;
#pragma unroll
    for (int t = 0; t < kFirst; ++t)
      if (t < ksteps) single_step(t, t);
    for (s = kFirst; s + kLoop + NS - 1 <= ksteps; s += kLoop) {
#pragma unroll
      for (int r = 0; r < kLoop / 4; ++r) {
        const StageSrc d = round_src();
#pragma unroll
        for (int j = 0; j < 4; ++j) phase_step(kFirst + 4 * r + j, d, j);
      }
    }
#pragma unroll
    for (int t = 0; t < kLoop + NS - 2; ++t)
      if (s + t < ksteps) single_step(kFirst + t, s + t);
  } else {
    const int32_t full = ksteps - ksteps % NS;
    for (; s < full; s += NS) {
#pragma unroll
      for (int j = 0; j < NS; ++j) single_step(j, s + j);
    }
#pragma unroll
    for (int j = 0; j < NS - 1; ++j)
      if (s + j < ksteps) single_step(j, s + j);
  }

  if (tl_on) {
    tl_rt[2] = __builtin_amdgcn_s_memrealtime();
    tl_clk[1] = __builtin_amdgcn_s_memtime();
  }
  static_assert((BM / 2) * BN * 2 <= NS * T::A_BYTES && (BM / 2) * BN * 2 <= NS * T::B_BYTES,
                "each half of the bf16 C tile fits in one operand's stage buffers");
  if (p.epi == 0 && !p.c_f32 && !p.ws)
    store_tile_staged<BM, BN, T::NW, T::TM, T::TN, T::WM, T::WN, true>(
        p, acc, &smA[0][0], &smB[0][0], pr, pc, ti, tj, wm, wn, wave, lane);
  else
    store_tile<BM, BN, 16, T::TM, T::TN, T::WM, T::WN>(p, acc, pr, pc, ti, tj, split, wm, wn, lane);
  if (tl_on) record_timeline(p.timeline + ((int64_t)blockIdx.x * T::NW + wave) * kTimelineWords,
                             tl_rt, tl_clk, lane);
#endif
}

// ---------------------------------------------------------------------------
// bf16 256x256 with whole-line A loads. The 32-K kernel fetches A as 64-byte
// half lines; here A is staged in 64-K pairs of steps (256 rows of 128
// bytes, chunk c of row r at c ^ swz_a64(r)), in a ring of three pair
// buffers (96 KiB), beside B's ring of four 32-K stages (64 KiB). Step s
// reads A from pair s / 2 (half s % 2) and B from stage s % 4; each step
// loads B for step s + 3 and every even step loads the A pair of steps
// s + 4, s + 5, into the buffer its steps s - 2, s - 1 left. A wave issues
// its A loads before its B loads, so at every stage barrier exactly 8 of
// its loads may stay in flight (those of the two previous steps' B and the
// current even step's A, or the previous even step's A and B and the
// current step's B). The MFMA schedule is the 32-K kernel's.
// ---------------------------------------------------------------------------

struct TileA2 {
  static constexpr int BM = 256, BN = 256, WGN = 4;
  static constexpr int NW = 8;
  static constexpr int THREADS = 64 * NW;
  static constexpr int WM = BM / 2, WN = BN / WGN;     // wave tile 128 x 64
  static constexpr int TM = WM / 16, TN = WN / 16;
  static constexpr int A2_BYTES = BM * 128;            // one pair of K steps
  static constexpr int B_BYTES = kBK * BN * 2;         // one 32-K stage
  static constexpr int NP = 3;                         // A pair buffers
  static constexpr int NSB = 4;                        // B stages
  static constexpr int NAP = A2_BYTES / (1024 * NW);   // A loads per wave per pair
  static constexpr int CPR_B = BN / 8;
  static constexpr int RPI_B = 64 / CPR_B;
  static constexpr int NB = B_BYTES / (1024 * NW);     // B loads per wave per step
  static_assert(NP * A2_BYTES + NSB * B_BYTES <= 160 * 1024, "LDS exceeds 160 KiB");
  static_assert(NAP == 4 && NB == 2, "the stage wait count below assumes 4 + 2 loads");
};

// Column tile of the j-th MFMA in tile row mt of a step: the rows are
// walked in a snake (odd rows right to left), so that consecutive MFMAs of
// a wave change one operand fragment, never both. Every accumulator still
// takes its K steps in order (same bits). Same box, alternating processes,
// 1400 W: +0.3-0.8 % TFLOP/s and a ~10 MHz higher sustained clock on the
// Llama FFN GEMMs.
template <int TN>
__device__ __forceinline__ constexpr int a2_nt(int mt, int j) {
  return (mt & 1) ? TN - 1 - j : j;
}

__global__ void __launch_bounds__(512, 2) gemm_a2_kernel(GemmParams p) {
#if defined(__HIP_DEVICE_COMPILE__)
  using T = TileA2;
  constexpr int BM = T::BM, BN = T::BN;
  __shared__ __attribute__((aligned(1024))) char smA[T::NP][T::A2_BYTES];
  __shared__ __attribute__((aligned(1024))) char smB[T::NSB][T::B_BYTES];

  const bool tl_on = p.timeline != nullptr;
  uint64_t tl_rt[3] = {0, 0, 0}, tl_clk[2] = {0, 0};
  if (tl_on) {
    tl_rt[0] = __builtin_amdgcn_s_memrealtime();
    tl_clk[0] = __builtin_amdgcn_s_memtime();
  }
  int32_t pr, pc, ti, tj, split;
  if (!tile_of_block(p, &pr, &pc, &ti, &tj, &split)) return;
  const int32_t ksteps = p.ksteps;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / T::WGN, wn = wave % T::WGN;

  uint32_t a_voff[T::NAP];
#pragma unroll
  for (int i = 0; i < T::NAP; ++i) {
    const int row = 8 * (wave * T::NAP + i) + (lane >> 3);
    const int chunk = (lane & 7) ^ swz_a64(row);
    // minus the instruction offset 1024 i of load i in its run (row >= 8 i
    // and ld >= 64, so the difference stays non-negative)
    a_voff[i] = (uint32_t)(row * p.a.ld + chunk * 8) * 2u - 1024u * i;
  }
  uint32_t b_voff[T::NB];
#pragma unroll
  for (int i = 0; i < T::NB; ++i) {
    const int row = T::RPI_B * (wave * T::NB + i) + lane / T::CPR_B;
    const int chunk = (lane % T::CPR_B) ^ swz_b(row);
    b_voff[i] = (uint32_t)(row * p.b.ld + chunk * 8) * 2u - 1024u * i;   // row >= 2 i, ld >= 256
  }
  // A: one descriptor for the tile's 256 rows over all K blocks of the
  // operand (the launch checks that it fits in 31 bits); the scalar offset
  // selects the pair.
  const int32_t a_blocks = p.ksteps * kBK / p.a.kslice;
  const int32_t a_extent = (a_blocks - 1) * p.a.slice * 2 + (BM - 1) * p.a.ld * 2 + p.a.kslice * 2;
  const int32_t b_extent = (kBK - 1) * p.b.ld * 2 + BN * 2;

  int32_t a_rd[2];
  {
    const int row = wm * T::WM + (lane & 15);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
      a_rd[kk] = row * 128 + (((4 * kk + (lane >> 4)) ^ swz_a64(row)) * 16);
  }
  int32_t b_rd[T::TN][2];
  {
    const int g = lane >> 4, s4 = lane & 15;
#pragma unroll
    for (int nt = 0; nt < T::TN; ++nt) {
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int krow = 8 * g + 4 * r + (s4 >> 2);
        const int col = wn * T::WN + nt * 16 + 4 * (s4 & 3);
        b_rd[nt][r] = krow * (BN * 2) + (((col >> 3) ^ swz_b(krow)) * 16) + ((col >> 2) & 1) * 8;
      }
    }
  }

  // ---- operand corners. A advances one pair (64 K) at a time, B one step ----
  const uint16_t* a_base = p.A + pr * p.a.part + (int64_t)(ti * BM) * p.a.ld;
  const uint16_t* b_base = p.B + pc * p.b.part + tj * BN;
  const char* b_next = reinterpret_cast<const char*>(b_base);
  const int32_t a_pairs = p.a.kslice / 64, b_steps = p.b.kslice / kBK;
  int32_t a_left = a_pairs, b_left = b_steps;
  // scalar offset from one pair to the next, and from the last pair of a K
  // block to the first of the next
  const uint32_t a_adv = 128u, a_adv_wrap = 128u + (uint32_t)(p.a.slice - p.a.kslice) * 2u;
  const int64_t b_adv = (int64_t)kBK * p.b.ld * 2;
  const int64_t b_jump = (p.b.slice - (int64_t)p.b.kslice * p.b.ld) * 2;
  const i32x4 a_desc = buffer_rsrc(a_base, a_extent);
  uint32_t a_so = 0;
  struct PairSrc {
    i32x4 r;
    uint32_t so;
  };
  // The next pair: the descriptor (empty past the last step, so no memory
  // is touched) and the pair's byte offset from the tile's first row.
  auto pair_src = [&](bool live) {
    PairSrc d;
    d.r = a_desc;
    if (!live) d.r[2] = 0;
    d.so = a_so;
    const bool wrap = --a_left == 0;
    a_so += wrap ? a_adv_wrap : a_adv;
    a_left = wrap ? a_pairs : a_left;
    return d;
  };
  auto b_src = [&](bool live) {
    const i32x4 r = buffer_rsrc(b_next, live ? b_extent : 0);
    const bool wrap = --b_left == 0;
    b_next += b_adv + (wrap ? b_jump : 0);
    b_left = wrap ? b_steps : b_left;
    return r;
  };
  const int32_t b_extent4 = (4 * kBK - 1) * p.b.ld * 2 + BN * 2;
  const uint32_t so_b[4] = {0u, (uint32_t)b_adv, (uint32_t)(2 * b_adv), (uint32_t)(3 * b_adv)};
  auto b_round_src = [&]() {
    const i32x4 r = buffer_rsrc(b_next, b_extent4);
    const bool wrap = b_left == 4;
    b_next += 4 * b_adv + (wrap ? b_jump : 0);
    b_left = wrap ? b_steps : b_left - 4;
    return r;
  };
  // Memory op i of a step's first half: A loads (i < NAP, even steps), then
  // B loads. A wave's loads of one operand in one step form a run sharing
  // M0 (LDS rows 1 KiB apart, 1024 i in the instruction offset).
  auto load_a = [&](const PairSrc& ra, char* dstA, int i) {
    if (i == 0) lds_dma16_first(ra.r, a_voff[0], ra.so, dstA + wave * T::NAP * 1024);
    else if (i == 1) lds_dma16_next<1024>(ra.r, a_voff[1], ra.so);
    else if (i == 2) lds_dma16_next<2048>(ra.r, a_voff[2], ra.so);
    else lds_dma16_next<3072>(ra.r, a_voff[3], ra.so);
  };
  auto load_b = [&](const i32x4& rb, int j, char* dstB, int i) {
    const uint32_t so = j < 0 ? 0u : so_b[j];
    if (i == 0) lds_dma16_first(rb, b_voff[0], so, dstB + wave * T::NB * 1024);
    else lds_dma16_next<1024>(rb, b_voff[1], so);
  };

  constexpr int kHalfM = T::TM / 2;
  AFrags<T::TM> fa;
  BFrags<T::TN> fb0, fb1;
  auto read_a = [&](const char* sA, int kk, int mt) {
    fa.a[mt] = *(const lds_bf16x8*)(sA + a_rd[kk] + mt * 16 * 128);
  };
  auto read_b = [&](const char* sB, BFrags<T::TN>& fb, int i) {
    const int nt = i >> 1, r = i & 1;
    fb.b[nt][r] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(sB + b_rd[nt][r]));
  };
  f32x4 acc[T::TM][T::TN];
#pragma unroll
  for (int i = 0; i < T::TM; ++i)
#pragma unroll
    for (int j = 0; j < T::TN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[i][j][v] = 0.f;
  auto mfma_one = [&](const BFrags<T::TN>& fb, int mt, int nt) {
    const bf16x8 bv = __builtin_bit_cast(
        bf16x8, __builtin_shufflevector(fb.b[nt][0], fb.b[nt][1], 0, 1, 2, 3, 4, 5, 6, 7));
    acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bv, fa.a[mt], acc[mt][nt], 0, 0, 0);
  };
  auto stage_barrier = [&]() {
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(8, 0));
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  // One step: A half kk of pair buffer sA, B stage sB; fragments of the
  // next step from (nA, nkk) and nB. With LA the step loads the A pair
  // (descriptor ra) into lA; B loads for step + 3 go to lB.
  auto step = [&](auto LA, const char* sA, int kk, const char* sB, const BFrags<T::TN>& fb,
                  BFrags<T::TN>& fbn, char* lA, const PairSrc& ra, char* lB, const i32x4& rb, int j,
                  const char* nA, int nkk, const char* nB) {
    constexpr bool kLoadA = decltype(LA)::value;
    constexpr int kMfmaHalf = kHalfM * T::TN;
    constexpr int kNA = kLoadA ? T::NAP : 0;
    constexpr int kOps1 = kHalfM + kNA + T::NB;
#pragma unroll
    for (int i = 0; i < kMfmaHalf; ++i) {
      mfma_one(fb, i / T::TN, a2_nt<T::TN>(i / T::TN, i % T::TN));
      if (i < kHalfM) read_a(sA, kk, kHalfM + i);
      else if (i < kHalfM + kNA) load_a(ra, lA, i - kHalfM);
      else if (i < kOps1) load_b(rb, j, lB, i - kHalfM - kNA);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = kMfmaHalf; i < kOps1; ++i) {
      if (i < kHalfM) read_a(sA, kk, kHalfM + i);
      else if (i < kHalfM + kNA) load_a(ra, lA, i - kHalfM);
      else load_b(rb, j, lB, i - kHalfM - kNA);
    }
    __builtin_amdgcn_sched_barrier(0);
    stage_barrier();
    constexpr int kOps2 = kHalfM + 2 * T::TN;
#pragma unroll
    for (int i = 0; i < kMfmaHalf; ++i) {
      mfma_one(fb, kHalfM + i / T::TN, a2_nt<T::TN>(kHalfM + i / T::TN, i % T::TN));
      if (i < kHalfM) read_a(nA, nkk, i);
      else if (i < kOps2) read_b(nB, fbn, i - kHalfM);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = kMfmaHalf; i < kOps2; ++i) {
      if (i < kHalfM) read_a(nA, nkk, i);
      else read_b(nB, fbn, i - kHalfM);
    }
    __builtin_amdgcn_sched_barrier(0);
  };

  // Prologue, in the order the steady state issues them: A pair 0, B 0,
  // A pair 1, B 1, B 2; then A pair 0 and B 0 complete.
  {
    const PairSrc r0 = pair_src(0 < ksteps);
#pragma unroll
    for (int i = 0; i < T::NAP; ++i) load_a(r0, smA[0], i);
    const i32x4 b0 = b_src(0 < ksteps);
#pragma unroll
    for (int i = 0; i < T::NB; ++i) load_b(b0, -1, smB[0], i);
    const PairSrc r1 = pair_src(2 < ksteps);
#pragma unroll
    for (int i = 0; i < T::NAP; ++i) load_a(r1, smA[1], i);
    const i32x4 b1 = b_src(1 < ksteps);
#pragma unroll
    for (int i = 0; i < T::NB; ++i) load_b(b1, -1, smB[1], i);
    const i32x4 b2 = b_src(2 < ksteps);
#pragma unroll
    for (int i = 0; i < T::NB; ++i) load_b(b2, -1, smB[2], i);
  }
  stage_barrier();
  if (tl_on) tl_rt[1] = __builtin_amdgcn_s_memrealtime();
#pragma unroll
  for (int mt = 0; mt < kHalfM; ++mt) read_a(smA[0], 0, mt);
#pragma unroll
  for (int i = 0; i < 2 * T::TN; ++i) read_b(smB[0], fb0, i);

  // Step s (phase ph = s mod 12): A pair buffer (s / 2) % 3, half s % 2; B
  // stage s % 4; even steps load the A pair s / 2 + 2 into buffer
  // (s / 2 + 2) % 3; B loads of step s + 3 into stage (s + 3) % 4.
  auto phase_step = [&](auto PH, const i32x4& rb, int j, int32_t s) {
    constexpr int ph = decltype(PH)::value;
    constexpr bool even = ph % 2 == 0;
    // inside the rounds loop (j >= 0) every pair it loads is live
    PairSrc ra = {};
    if constexpr (even) ra = pair_src(j >= 0 || 2 * (s / 2 + 2) < ksteps);
    step(std::integral_constant<bool, even>{}, smA[(ph / 2) % 3], ph % 2, smB[ph % 4],
         ph % 2 ? fb1 : fb0, ph % 2 ? fb0 : fb1, smA[(ph / 2 + 2) % 3], ra, smB[(ph + 3) % 4], rb,
         j, smA[((ph + 1) / 2) % 3], (ph + 1) % 2, smB[(ph + 1) % 4]);
  };
  auto single_step = [&](auto PH, int32_t s) {
    const i32x4 rb = b_src(s + 3 < ksteps);
    phase_step(PH, rb, -1, s);
  };
  int32_t s = 0;
  if (p.round_fast) {
    // Step 0 alone; rounds of 4 B-steps (s = 1 mod 4) whose B loads share
    // one descriptor; 12 steps per loop iteration so that every phase is a
    // compile-time constant, each loading only live A pairs (the last, at
    // step s + 11, covers steps s + 15 and s + 16) and B stages; the
    // remaining steps (at most 15) alone.
    single_step(std::integral_constant<int, 0>{}, 0);
    for (s = 1; s + 16 <= ksteps; s += 12) {
      const i32x4 rb0 = b_round_src();
      phase_step(std::integral_constant<int, 1>{}, rb0, 0, s);
      phase_step(std::integral_constant<int, 2>{}, rb0, 1, s + 1);
      phase_step(std::integral_constant<int, 3>{}, rb0, 2, s + 2);
      phase_step(std::integral_constant<int, 4>{}, rb0, 3, s + 3);
      const i32x4 rb1 = b_round_src();
      phase_step(std::integral_constant<int, 5>{}, rb1, 0, s + 4);
      phase_step(std::integral_constant<int, 6>{}, rb1, 1, s + 5);
      phase_step(std::integral_constant<int, 7>{}, rb1, 2, s + 6);
      phase_step(std::integral_constant<int, 8>{}, rb1, 3, s + 7);
      const i32x4 rb2 = b_round_src();
      phase_step(std::integral_constant<int, 9>{}, rb2, 0, s + 8);
      phase_step(std::integral_constant<int, 10>{}, rb2, 1, s + 9);
      phase_step(std::integral_constant<int, 11>{}, rb2, 2, s + 10);
      phase_step(std::integral_constant<int, 12>{}, rb2, 3, s + 11);
    }
#define CCL_A2_TAIL(t) if (s + (t) < ksteps) single_step(std::integral_constant<int, 1 + (t)>{}, s + (t))
    CCL_A2_TAIL(0); CCL_A2_TAIL(1); CCL_A2_TAIL(2); CCL_A2_TAIL(3); CCL_A2_TAIL(4);
    CCL_A2_TAIL(5); CCL_A2_TAIL(6); CCL_A2_TAIL(7); CCL_A2_TAIL(8); CCL_A2_TAIL(9);
    CCL_A2_TAIL(10); CCL_A2_TAIL(11); CCL_A2_TAIL(12); CCL_A2_TAIL(13); CCL_A2_TAIL(14);
#undef CCL_A2_TAIL
  } else {
    for (; s + 12 <= ksteps; s += 12) {
#define CCL_A2_STEP(t) single_step(std::integral_constant<int, (t)>{}, s + (t))
      CCL_A2_STEP(0); CCL_A2_STEP(1); CCL_A2_STEP(2); CCL_A2_STEP(3); CCL_A2_STEP(4); CCL_A2_STEP(5);
      CCL_A2_STEP(6); CCL_A2_STEP(7); CCL_A2_STEP(8); CCL_A2_STEP(9); CCL_A2_STEP(10); CCL_A2_STEP(11);
#undef CCL_A2_STEP
    }
#define CCL_A2_REST(t) if (s + (t) < ksteps) single_step(std::integral_constant<int, (t)>{}, s + (t))
    CCL_A2_REST(0); CCL_A2_REST(1); CCL_A2_REST(2); CCL_A2_REST(3); CCL_A2_REST(4); CCL_A2_REST(5);
    CCL_A2_REST(6); CCL_A2_REST(7); CCL_A2_REST(8); CCL_A2_REST(9); CCL_A2_REST(10);
#undef CCL_A2_REST
  }

  if (tl_on) {
    tl_rt[2] = __builtin_amdgcn_s_memrealtime();
    tl_clk[1] = __builtin_amdgcn_s_memtime();
  }
  static_assert((BM / 2) * BN * 2 <= T::NP * T::A2_BYTES && (BM / 2) * BN * 2 <= T::NSB * T::B_BYTES,
                "each half of the bf16 C tile fits in one operand's buffers");
  if (p.epi == 0 && !p.c_f32 && !p.ws)
    store_tile_staged<BM, BN, T::NW, T::TM, T::TN, T::WM, T::WN>(p, acc, &smA[0][0], &smB[0][0], pr,
                                                                 pc, ti, tj, wm, wn, wave, lane);
  else
    store_tile<BM, BN, 16, T::TM, T::TN, T::WM, T::WN>(p, acc, pr, pc, ti, tj, split, wm, wn, lane);
  if (tl_on) record_timeline(p.timeline + ((int64_t)blockIdx.x * T::NW + wave) * kTimelineWords,
                             tl_rt, tl_clk, lane);
#endif
}

// ---------------------------------------------------------------------------
// fp8 (E4M3) operands: C = A B with v_mfma_f32_32x32x64_f8f6f4 (unscaled).
// A K step is 64 fp8 elements, so one stage holds the same bytes as a bf16
// step (A rows of 64 bytes, B rows of BN bytes x 64 rows) and the A side
// (loads, swizzle, fragment reads) is byte-for-byte the bf16 one.
//
// Operand pairing of the instruction (probed on gfx950): byte p of lane l in
// the first operand meets byte p of lanes of the same half (l / 32) in the
// second, and lane l % 32 selects the row / column. The K index of (half h,
// byte p) is chosen here as 16h + p for p < 16 and 32 + 16h + (p - 16) for
// p >= 16: the A fragment is then the two 16-byte chunks h and 2 + h of a
// 64-byte row, as in the bf16 kernel, and the B fragment is four transposed
// 8-byte reads (ds_read_b64_tr_b8: within 16 lanes, lane l, byte j comes
// from source lane 2j + l/8, byte l % 8), each giving 8 consecutive K of one
// column.
// ---------------------------------------------------------------------------

constexpr int kBK8 = 64;         // K extent (elements = bytes) of one fp8 step

typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4v __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) i32x2 lds_i32x2;
typedef __attribute__((address_space(3))) i32x4v lds_i32x4;

template <int BM, int BN, int WGN>
struct Tile8 {
  static constexpr int NW = 2 * WGN;
  static constexpr int THREADS = 64 * NW;
  static constexpr int WM = BM / 2, WN = BN / WGN;
  static constexpr int TM = WM / 32, TN = WN / 32;
  static constexpr int A_BYTES = BM * kBK8;            // one stage
  static constexpr int B_BYTES = kBK8 * BN;
  static constexpr int NA = BM / (16 * NW);            // A: 16 rows of 64 B per load
  static constexpr int CPR_B = BN / 16;                // 16-byte chunks per B row
  static constexpr int RPI_B = 64 / CPR_B;             // B rows per load instruction
  static constexpr int NB = BN / (16 * NW);
  static constexpr int NL = NA + NB;
  static_assert(NA >= 1 && NB >= 1 && TN >= 1, "tile too small for the wave grid");
  static_assert(BN == 128 || BN == 256, "B swizzle is defined for 128- and 256-byte rows");
};

// B rows (BN bytes): the 8 rows x 2 chunks that 32 lanes of one transposed
// read touch land in 16 distinct 16-byte bank slots.
template <int BN>
__device__ __forceinline__ int swz_b8(int row) {
  return BN == 256 ? 2 * (row & 7) : (row & 6);
}

template <int TM, int TN>
struct FragSet8 {
  i32x8 a[TM];
  i32x8 b[TN];
};

template <int BM, int BN, int WGN>
__global__ void __launch_bounds__(128 * WGN, WGN / 2) gemm_fp8_kernel(GemmParams p) {
#if defined(__HIP_DEVICE_COMPILE__)
  using T = Tile8<BM, BN, WGN>;
  constexpr int NS = kStages;
  __shared__ __attribute__((aligned(1024))) char smA[NS][T::A_BYTES];
  __shared__ __attribute__((aligned(1024))) char smB[NS][T::B_BYTES];

  int32_t pr, pc, ti, tj, split;
  if (!tile_of_block(p, &pr, &pc, &ti, &tj, &split)) return;
  // K range of this workgroup: steps [k0, k0 + ksteps) (all of K without split-K)
  const int32_t k0 = __builtin_amdgcn_readfirstlane(split * p.ksteps_per_split);
  const int32_t ksteps = __builtin_amdgcn_readfirstlane(min(p.ksteps, k0 + p.ksteps_per_split) - k0);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  const char* A = reinterpret_cast<const char*>(p.A);
  const char* B = reinterpret_cast<const char*>(p.B);

  // ---- global -> LDS (byte offsets from the K step's tile corner) ----
  uint32_t a_voff[T::NA];
#pragma unroll
  for (int i = 0; i < T::NA; ++i) {
    const int row = 16 * (wave * T::NA + i) + (lane >> 2);
    const int chunk = (lane & 3) ^ swz_a(row);
    a_voff[i] = (uint32_t)(row * p.a.ld + chunk * 16);
  }
  uint32_t b_voff[T::NB];
#pragma unroll
  for (int i = 0; i < T::NB; ++i) {
    const int row = T::RPI_B * (wave * T::NB + i) + lane / T::CPR_B;
    const int chunk = (lane % T::CPR_B) ^ swz_b8<BN>(row);
    b_voff[i] = (uint32_t)(row * p.b.ld + chunk * 16);
  }
  const int32_t a_extent = (BM - 1) * p.a.ld + kBK8;
  const int32_t b_extent = (kBK8 - 1) * p.b.ld + BN;

  // ---- LDS fragment read offsets (bytes) ----
  int32_t a_rd[2];
  {
    const int row = wm * T::WM + (lane & 31);
    const int h = lane >> 5;
#pragma unroll
    for (int c = 0; c < 2; ++c) a_rd[c] = row * 64 + (((2 * c + h) ^ swz_a(row)) * 16);
  }
  int32_t b_rd[T::TN][4];
  {
    const int g = lane >> 4, s = lane & 15;
    const int h = g >> 1, cb = g & 1;
#pragma unroll
    for (int nt = 0; nt < T::TN; ++nt) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int kbase = (r < 2) ? 16 * h + 8 * r : 32 + 16 * h + 8 * (r - 2);
        const int krow = kbase + (s >> 1);
        const int col = wn * T::WN + nt * 32 + 16 * cb + 8 * (s & 1);
        b_rd[nt][r] = krow * BN + (((col >> 4) ^ swz_b8<BN>(krow)) * 16) + (col & 15);
      }
    }
  }

  const char* a_base = A + pr * p.a.part + (int64_t)(ti * BM) * p.a.ld;
  const char* b_base = B + pc * p.b.part + tj * BN;
  int64_t a_slice_off, b_slice_off;
  int32_t a_kl, b_kl;
  k_start(p.a, k0 * kBK8, &a_slice_off, &a_kl);
  k_start(p.b, k0 * kBK8, &b_slice_off, &b_kl);

  // Byte address of the next K step's A and B corners; one step at a time,
  // with a jump to the next CCL K block after a block's last step.
  const char* a_next = a_base + a_slice_off + a_kl;
  const char* b_next = b_base + b_slice_off + (int64_t)b_kl * p.b.ld;
  const int32_t a_steps = p.a.kslice / kBK8, b_steps = p.b.kslice / kBK8;   // steps per block
  int32_t a_left = a_steps - a_kl / kBK8, b_left = b_steps - b_kl / kBK8;   // left in this block
  const int64_t a_adv = kBK8, b_adv = (int64_t)kBK8 * p.b.ld;
  const int64_t a_jump = p.a.slice - p.a.kslice;
  const int64_t b_jump = p.b.slice - (int64_t)p.b.kslice * p.b.ld;

  // Descriptors of the next K step to be loaded. With live == false they
  // cover zero bytes: every load is out of range, touches no memory and
  // writes zeros to the (unused) stage.
  struct StageSrc {
    i32x4 ra, rb;
  };
  auto next_src = [&](bool live) {
    StageSrc d;
    d.ra = buffer_rsrc(a_next, live ? a_extent : 0);
    d.rb = buffer_rsrc(b_next, live ? b_extent : 0);
    const bool a_wrap = --a_left == 0;
    a_next += a_adv + (a_wrap ? a_jump : 0);
    a_left = a_wrap ? a_steps : a_left;
    const bool b_wrap = --b_left == 0;
    b_next += b_adv + (b_wrap ? b_jump : 0);
    b_left = b_wrap ? b_steps : b_left;
    return d;
  };
  auto load_one = [&](const StageSrc& d, char* sA, char* sB, int i) {
    if (i < T::NA)
      lds_dma16(d.ra, a_voff[i], sA + (wave * T::NA + i) * 1024);
    else
      lds_dma16(d.rb, b_voff[i - T::NA], sB + (wave * T::NB + (i - T::NA)) * 1024);
  };
  auto load_stage = [&](char* sA, char* sB, bool live) {
    const StageSrc d = next_src(live);
#pragma unroll
    for (int i = 0; i < T::NL; ++i) load_one(d, sA, sB, i);
  };

  using Frags = FragSet8<T::TM, T::TN>;
  // Reads of one stage's fragments: 2 per A tile (16-byte chunks), 4 per B
  // tile (8-byte transposed reads), A first.
  constexpr int kReads = 2 * T::TM + 4 * T::TN;
  auto read_one = [&](const char* smA, const char* smB, Frags& f, int i) {
    if (i < 2 * T::TM) {
      const int mt = i >> 1, c = i & 1;
      const i32x4v v = *(const lds_i32x4*)(smA + a_rd[c] + mt * 32 * 64);
#pragma unroll
      for (int j = 0; j < 4; ++j) f.a[mt][4 * c + j] = v[j];
    } else {
      const int nt = (i - 2 * T::TM) >> 2, r = (i - 2 * T::TM) & 3;
      const i32x2 v = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2*)(smB + b_rd[nt][r]));
      f.b[nt][2 * r] = v[0];
      f.b[nt][2 * r + 1] = v[1];
    }
  };
  auto read_frags = [&](const char* smA, const char* smB, Frags& f) {
#pragma unroll
    for (int i = 0; i < kReads; ++i) read_one(smA, smB, f, i);
  };

  f32x16 acc[T::TM][T::TN];
#pragma unroll
  for (int i = 0; i < T::TM; ++i)
#pragma unroll
    for (int j = 0; j < T::TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  constexpr int kMfma = T::TM * T::TN;
  constexpr int kHalf = (kMfma + 1) / 2;
  auto mfma_one = [&](const Frags& f, int i) {
    const int mt = i / T::TN, nt = i % T::TN;
    acc[mt][nt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(f.b[nt], f.a[mt], acc[mt][nt],
                                                                  0, 0, 0, 0, 0, 0);
  };
  auto stage_barrier = [&]() {
    __builtin_amdgcn_s_waitcnt(waitcnt_imm((kStages - 2) * T::NL, 0));
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  // One K step on the stage whose fragments are in f: the first half of the
  // MFMAs issues the loads of the step NS-1 ahead into (lA, lB) with the
  // descriptors d; after the barrier the second half
  // reads the next stage's (nA, nB) fragments into g. The fragment sets
  // alternate between steps.
  auto step = [&](const Frags& f, Frags& g, char* lA, char* lB, const char* nA, const char* nB,
                  const StageSrc& d) {
#pragma unroll
    for (int i = 0; i < kHalf; ++i) {
      mfma_one(f, i);
      const int per = (T::NL + kHalf - 1) / kHalf;
#pragma unroll
      for (int q = 0; q < per; ++q)
        if (i * per + q < T::NL) load_one(d, lA, lB, i * per + q);
      __builtin_amdgcn_sched_barrier(0);
    }
    stage_barrier();
    constexpr int rest = kMfma - kHalf;
    constexpr int per = rest > 0 ? (kReads + rest - 1) / rest : kReads;
#pragma unroll
    for (int i = 0; i < rest; ++i) {
      mfma_one(f, kHalf + i);
#pragma unroll
      for (int q = 0; q < per; ++q)
        if (i * per + q < kReads) read_one(nA, nB, g, i * per + q);
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (rest == 0) read_frags(nA, nB, g);
    __builtin_amdgcn_sched_barrier(0);
  };

  Frags f0, f1;
#pragma unroll
  for (int j = 0; j < NS - 1; ++j) load_stage(smA[j], smB[j], j < ksteps);
  stage_barrier();
  read_frags(smA[0], smB[0], f0);
  // Step s works on stage s % NS, loads stage (s + NS - 1) % NS and reads
  // stage (s + 1) % NS; ph is s modulo NS (a multiple of 2). Whole rounds of
  // NS steps run branch-free (so the compiler tracks the outstanding LDS
  // reads exactly); the last, partial round runs its steps under conditions.
  // (The bf16 kernel's rounds path, one descriptor per four steps, needs
  // more scalar registers than this kernel has left.)
  static_assert(NS % 2 == 0, "fragment sets alternate by step parity");
  auto single_step = [&](int ph, int32_t s) {
    const StageSrc d = next_src(s + NS - 1 < ksteps);
    step(ph % 2 ? f1 : f0, ph % 2 ? f0 : f1, smA[(ph + NS - 1) % NS], smB[(ph + NS - 1) % NS],
         smA[(ph + 1) % NS], smB[(ph + 1) % NS], d);
  };
  int32_t s = 0;
  const int32_t full = ksteps - ksteps % NS;
  for (; s < full; s += NS) {
#pragma unroll
    for (int j = 0; j < NS; ++j) single_step(j, s + j);
  }
#pragma unroll
  for (int j = 0; j < NS - 1; ++j)
    if (s + j < ksteps) single_step(j, s + j);

  store_tile<BM, BN, 32, T::TM, T::TN, T::WM, T::WN>(p, acc, pr, pc, ti, tj, split, wm, wn, lane);
#endif
}

// ---------------------------------------------------------------------------
// fp8 (E4M3) operands on v_mfma_f32_16x16x128_f8f6f4 (unscaled). One
// instruction covers a whole 128-wide K step, so a stage holds 128 K: A rows
// of 128 bytes and B rows of BN bytes x 128 rows, 64 KiB for a 256x256 tile.
// Two stages: the loads of step t+1 are issued at the start of step t,
// right after the barrier that frees their stage.
//
// K order inside an instruction: lane l (16-lane group g = l / 16) holds 32
// bytes; byte p < 16 is K = 16 g + p and byte p >= 16 is K = 64 + 16 g +
// (p - 16). A and B use the same order, so every product pairs equal K.
// A fragment: 16-byte chunks g and 4 + g of a 128-byte row (two
// ds_read_b128). B fragment: four ds_read_b64_tr_b8, rows 16 g + 8 r and
// 64 + 16 g + 8 r, each giving 8 consecutive K of the lane's column.
// ---------------------------------------------------------------------------

constexpr int kBK8x = 128;       // K extent of one step of gemm_fp8x_kernel

template <int BM, int BN, int WGN>
struct Tile8x {
  static constexpr int NW = 2 * WGN;
  static constexpr int THREADS = 64 * NW;
  static constexpr int WM = BM / 2, WN = BN / WGN;
  static constexpr int TM = WM / 16, TN = WN / 16;
  static constexpr int A_BYTES = BM * kBK8x;           // one stage
  static constexpr int B_BYTES = kBK8x * BN;
  static constexpr int NA = A_BYTES / (1024 * NW);     // 8 A rows of 128 B per load
  static constexpr int CPR_B = BN / 16;                // 16-byte chunks per B row
  static constexpr int RPI_B = 64 / CPR_B;             // B rows per load instruction
  static constexpr int NB = B_BYTES / (1024 * NW);
  static constexpr int NL = NA + NB;
  static_assert(NA >= 1 && NB >= 1 && TN >= 2 && TM >= 2, "tile too small for the wave grid");
  static_assert(BN == 128 || BN == 256, "B swizzle is defined for 128- and 256-byte rows");
  static_assert(TM * TN * 4 <= 128, "accumulators must fit in 128 VGPRs (two waves per SIMD)");
};

// Swizzles, conflict-free under the measured bank model: A (128-byte rows,
// 16 rows x 2 chunks per ds_read_b128 half-wave pair): chunk XOR (row & 6).
// B (BN-byte rows; a half-wave of one transposed read touches 16 rows x one
// 16-byte chunk): 256-byte rows XOR (row & 7) | 8 bit4(row); 128-byte rows
// XOR (row >> 1 & 3) | 4 bit4(row).
__device__ __forceinline__ int swz_a8x(int row) { return row & 6; }
template <int BN>
__device__ __forceinline__ int swz_b8x(int row) {
  return BN == 256 ? ((row & 7) | (((row >> 4) & 1) << 3)) : (((row >> 1) & 3) | (((row >> 4) & 1) << 2));
}

template <int BM, int BN, int WGN>
__global__ void __launch_bounds__(128 * WGN, WGN / 2) gemm_fp8x_kernel(GemmParams p) {
#if defined(__HIP_DEVICE_COMPILE__)
  using T = Tile8x<BM, BN, WGN>;
  __shared__ __attribute__((aligned(1024))) char smA[2][T::A_BYTES];
  __shared__ __attribute__((aligned(1024))) char smB[2][T::B_BYTES];

  int32_t pr, pc, ti, tj, split;
  if (!tile_of_block(p, &pr, &pc, &ti, &tj, &split)) return;
  const int32_t k0 = __builtin_amdgcn_readfirstlane(split * p.ksteps_per_split);
  const int32_t ksteps = __builtin_amdgcn_readfirstlane(min(p.ksteps, k0 + p.ksteps_per_split) - k0);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;

  // ---- global -> LDS (byte offsets from the K step's tile corner) ----
  uint32_t a_voff[T::NA];
#pragma unroll
  for (int i = 0; i < T::NA; ++i) {
    const int row = 8 * (wave * T::NA + i) + (lane >> 3);
    const int chunk = (lane & 7) ^ swz_a8x(row);
    a_voff[i] = (uint32_t)(row * p.a.ld + chunk * 16);
  }
  uint32_t b_voff[T::NB];
#pragma unroll
  for (int i = 0; i < T::NB; ++i) {
    const int row = T::RPI_B * (wave * T::NB + i) + lane / T::CPR_B;
    const int chunk = (lane % T::CPR_B) ^ swz_b8x<BN>(row);
    b_voff[i] = (uint32_t)(row * p.b.ld + chunk * 16);
  }
  const int32_t a_extent = (BM - 1) * p.a.ld + kBK8x;
  const int32_t b_extent = (kBK8x - 1) * p.b.ld + BN;

  // ---- LDS fragment read offsets (bytes); A tile mt adds mt * 16 rows ----
  int32_t a_rd[2];
  {
    const int row = wm * T::WM + (lane & 15);
    const int g = lane >> 4;
#pragma unroll
    for (int h = 0; h < 2; ++h) a_rd[h] = row * kBK8x + (((4 * h + g) ^ swz_a8x(row)) * 16);
  }
  int32_t b_rd[T::TN][4];
  {
    const int g = lane >> 4, s = lane & 15;
#pragma unroll
    for (int nt = 0; nt < T::TN; ++nt) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int krow = 64 * (r >> 1) + 16 * g + 8 * (r & 1) + (s >> 1);
        const int col = wn * T::WN + nt * 16 + 8 * (s & 1);
        b_rd[nt][r] = krow * BN + (((col >> 4) ^ swz_b8x<BN>(krow)) * 16) + (col & 15);
      }
    }
  }

  // ---- operand corners (see the bf16 kernel) ----
  const char* A = reinterpret_cast<const char*>(p.A);
  const char* B = reinterpret_cast<const char*>(p.B);
  const char* a_base = A + pr * p.a.part + (int64_t)(ti * BM) * p.a.ld;
  const char* b_base = B + pc * p.b.part + tj * BN;
  int64_t a_slice_off, b_slice_off;
  int32_t a_kl, b_kl;
  k_start(p.a, k0 * kBK8x, &a_slice_off, &a_kl);
  k_start(p.b, k0 * kBK8x, &b_slice_off, &b_kl);
  const char* a_next = a_base + a_slice_off + a_kl;
  const char* b_next = b_base + b_slice_off + (int64_t)b_kl * p.b.ld;
  const int32_t a_steps = p.a.kslice / kBK8x, b_steps = p.b.kslice / kBK8x;
  int32_t a_left = a_steps - a_kl / kBK8x, b_left = b_steps - b_kl / kBK8x;
  const int64_t a_adv = kBK8x, b_adv = (int64_t)kBK8x * p.b.ld;
  const int64_t a_jump = p.a.slice - p.a.kslice;
  const int64_t b_jump = p.b.slice - (int64_t)p.b.kslice * p.b.ld;
  struct StageSrc {
    i32x4 ra, rb;
  };
  auto next_src = [&](bool live) {
    StageSrc d;
    d.ra = buffer_rsrc(a_next, live ? a_extent : 0);
    d.rb = buffer_rsrc(b_next, live ? b_extent : 0);
    const bool a_wrap = --a_left == 0;
    a_next += a_adv + (a_wrap ? a_jump : 0);
    a_left = a_wrap ? a_steps : a_left;
    const bool b_wrap = --b_left == 0;
    b_next += b_adv + (b_wrap ? b_jump : 0);
    b_left = b_wrap ? b_steps : b_left;
    return d;
  };
  auto load_one = [&](const StageSrc& d, char* sA, char* sB, int i) {
    if (i < T::NA)
      lds_dma16(d.ra, a_voff[i], sA + (wave * T::NA + i) * 1024);
    else
      lds_dma16(d.rb, b_voff[i - T::NA], sB + (wave * T::NB + (i - T::NA)) * 1024);
  };

  i32x8 fa[2];             // A fragments of tiles mt (fa[mt % 2]) and mt + 1
  i32x8 fb[T::TN];
  auto read_a_half = [&](const char* sA, int mt, int h, i32x8& f) {
    const i32x4v v = *(const lds_i32x4*)(sA + a_rd[h] + mt * 16 * kBK8x);
#pragma unroll
    for (int q = 0; q < 4; ++q) f[4 * h + q] = v[q];
  };
  auto read_b = [&](const char* sB, int i) {     // i = 4 nt + r
    const int nt = i >> 2, r = i & 3;
    const i32x2 v = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2*)(sB + b_rd[nt][r]));
    fb[nt][2 * r] = v[0];
    fb[nt][2 * r + 1] = v[1];
  };

  f32x4 acc[T::TM][T::TN];
#pragma unroll
  for (int i = 0; i < T::TM; ++i)
#pragma unroll
    for (int j = 0; j < T::TN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[i][j][v] = 0.f;

  // Wait for the own loads of this step's stage, then for every wave: the
  // stage is complete in LDS and nobody still reads the other stage.
  auto step_barrier = [&]() {
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 0));
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  // One K step on stage st: first the loads of step t+1 into stage st ^ 1
  // (a whole step before they are needed), interleaved with the reads of
  // A tile 0 and all B fragments; then the MFMAs tile row by tile row, with
  // the reads of the next A tile (into the other A buffer) behind them.
  auto step = [&](int st, bool live_next) {
    const StageSrc d = next_src(live_next);
    const char* sA = smA[st];
    const char* sB = smB[st];
    constexpr int kFirst = 2 + 4 * T::TN;          // reads before the first MFMA
#pragma unroll
    for (int i = 0; i < (kFirst > T::NL ? kFirst : T::NL); ++i) {
      if (i < T::NL) load_one(d, smA[st ^ 1], smB[st ^ 1], i);
      if (i < 2) read_a_half(sA, 0, i, fa[0]);
      else if (i < kFirst) read_b(sB, i - 2);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int mt = 0; mt < T::TM; ++mt) {
#pragma unroll
      for (int nt = 0; nt < T::TN; ++nt) {
        acc[mt][nt] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(fb[nt], fa[mt & 1], acc[mt][nt],
                                                                       0, 0, 0, 0, 0, 0);
        if (nt < 2 && mt + 1 < T::TM) read_a_half(sA, mt + 1, nt, fa[(mt + 1) & 1]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };

  {
    const StageSrc d = next_src(0 < ksteps);
#pragma unroll
    for (int i = 0; i < T::NL; ++i) load_one(d, smA[0], smB[0], i);
  }
  // Steps in pairs (stages 0, 1) branch-free, then a last odd step.
  int32_t t = 0;
  for (; t + 2 <= ksteps; t += 2) {
    step_barrier();
    step(0, t + 1 < ksteps);
    step_barrier();
    step(1, t + 2 < ksteps);
  }
  if (t < ksteps) {
    step_barrier();
    step(0, false);
  }

  static_assert((BM / 2) * BN * 2 <= 2 * T::A_BYTES && (BM / 2) * BN * 2 <= 2 * T::B_BYTES,
                "each half of the bf16 C tile fits in one operand's stage buffers");
  if (p.epi == 0 && !p.c_f32 && !p.ws)
    store_tile_staged<BM, BN, T::NW, T::TM, T::TN, T::WM, T::WN>(p, acc, &smA[0][0], &smB[0][0], pr,
                                                                 pc, ti, tj, wm, wn, wave, lane);
  else
    store_tile<BM, BN, 16, T::TM, T::TN, T::WM, T::WN>(p, acc, pr, pc, ti, tj, split, wm, wn, lane);
#endif
}

// ---------------------------------------------------------------------------
// fp8 256x256 with the fragment reads pipelined across steps
// (gemm_fp8p_kernel). Same MFMA (16x16x128), K order, fragment layout and
// swizzles as gemm_fp8x_kernel, so every accumulator takes the same MFMAs
// in the same order and C is identical bit for bit; what changes is when
// loads and fragment reads are issued.
//
// gemm_fp8x_kernel opens every 128-K step with a barrier that waits for all
// of the step's loads, then issues the next step's loads and 18 fragment
// reads before its first MFMA: the matrix cores wait on that at every step.
// Here A has three 32 KiB stage buffers and B two (160 KiB), and a step
// (8 rows of 4 MFMAs per wave, snake order) has two barriers:
//  * after row 0 (X): every wave has read all of stage t's B fragments and
//    all of stage t-1's A, so the loads of stage t+2 (A into buffer
//    (t+2) % 3, B into (t+2) % 2) go out in rows 1-2;
//  * after row 5 (Y): stage t+1 is complete (its loads went out a step
//    earlier; only stage t+2's may still be in flight), so rows 6-7 read
//    stage t+1's B fragments (tiles 0-1 into two spare fragments, tiles 3
//    and 2 into the registers of the current ones right after their last
//    MFMA) and its A tile 0, behind the MFMAs.
// The next step's first MFMAs thus find their fragments in registers. The
// B fragment registers rotate with step parity (the loop runs step pairs).
// ---------------------------------------------------------------------------

struct TileFp8P {
  static constexpr int BM = 256, BN = 256, WGN = 4;
  static constexpr int NW = 8;
  static constexpr int THREADS = 64 * NW;
  static constexpr int WM = BM / 2, WN = BN / WGN;     // wave tile 128 x 64
  static constexpr int TM = WM / 16, TN = WN / 16;     // 8 x 4 MFMA tiles
  static constexpr int A_BYTES = BM * kBK8x;           // one stage
  static constexpr int B_BYTES = kBK8x * BN;
  static constexpr int NSA = 3, NSB = 2;
  static constexpr int NA = A_BYTES / (1024 * NW);     // 4 A loads per wave per stage
  static constexpr int CPR_B = BN / 16;
  static constexpr int RPI_B = 64 / CPR_B;
  static constexpr int NB = B_BYTES / (1024 * NW);     // 4 B loads per wave per stage
  static constexpr int NL = NA + NB;
  static constexpr int ROW_X = 0, ROW_Y = 5;           // rows followed by a barrier
  static_assert(NSA * A_BYTES + NSB * B_BYTES <= 160 * 1024, "LDS exceeds 160 KiB");
  static_assert(TM == 8 && TN == 4, "the row schedule below is written for 8 x 4 MFMA tiles");
};

__global__ void __launch_bounds__(512, 2) gemm_fp8p_kernel(GemmParams p) {
#if defined(__HIP_DEVICE_COMPILE__)
  using T = TileFp8P;
  constexpr int BM = T::BM, BN = T::BN;
  __shared__ __attribute__((aligned(1024))) char smA[T::NSA][T::A_BYTES];
  __shared__ __attribute__((aligned(1024))) char smB[T::NSB][T::B_BYTES];

  int32_t pr, pc, ti, tj, split;
  if (!tile_of_block(p, &pr, &pc, &ti, &tj, &split)) return;
  const int32_t ksteps = p.ksteps;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / T::WGN, wn = wave % T::WGN;

  uint32_t a_voff[T::NA];
#pragma unroll
  for (int i = 0; i < T::NA; ++i) {
    const int row = 8 * (wave * T::NA + i) + (lane >> 3);
    const int chunk = (lane & 7) ^ swz_a8x(row);
    // minus the instruction offset 1024 i of load i in its run (row >= 8 i,
    // ld >= 128)
    a_voff[i] = (uint32_t)(row * p.a.ld + chunk * 16) - 1024u * i;
  }
  uint32_t b_voff[T::NB];
#pragma unroll
  for (int i = 0; i < T::NB; ++i) {
    const int row = T::RPI_B * (wave * T::NB + i) + lane / T::CPR_B;
    const int chunk = (lane % T::CPR_B) ^ swz_b8x<BN>(row);
    b_voff[i] = (uint32_t)(row * p.b.ld + chunk * 16) - 1024u * i;   // row >= 4 i, ld >= 256
  }
  // One descriptor per operand for the whole tile: A's 256 rows and B's
  // 256 columns over all K blocks (the launch checks that both extents fit
  // in 31 bits); a stage is selected by the loads' scalar offset.
  const int32_t K = p.ksteps * kBK8x;
  const int32_t a_extent = (K / p.a.kslice - 1) * p.a.slice + (BM - 1) * p.a.ld + p.a.kslice;
  const int32_t b_extent = (int32_t)((K / p.b.kslice - 1) * p.b.slice +
                                     (int64_t)(p.b.kslice - 1) * p.b.ld + BN);

  int32_t a_rd[2];
  {
    const int row = wm * T::WM + (lane & 15);
    const int g = lane >> 4;
#pragma unroll
    for (int h = 0; h < 2; ++h) a_rd[h] = row * kBK8x + (((4 * h + g) ^ swz_a8x(row)) * 16);
  }
  int32_t b_rd[T::TN][4];
  {
    const int g = lane >> 4, s = lane & 15;
#pragma unroll
    for (int nt = 0; nt < T::TN; ++nt) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int krow = 64 * (r >> 1) + 16 * g + 8 * (r & 1) + (s >> 1);
        const int col = wn * T::WN + nt * 16 + 8 * (s & 1);
        b_rd[nt][r] = krow * BN + (((col >> 4) ^ swz_b8x<BN>(krow)) * 16) + (col & 15);
      }
    }
  }

  const char* A = reinterpret_cast<const char*>(p.A);
  const char* B = reinterpret_cast<const char*>(p.B);
  const i32x4 a_desc = buffer_rsrc(A + pr * p.a.part + (int64_t)(ti * BM) * p.a.ld, a_extent);
  const i32x4 b_desc = buffer_rsrc(B + pc * p.b.part + tj * BN, b_extent);
  const int32_t a_steps = p.a.kslice / kBK8x, b_steps = p.b.kslice / kBK8x;
  int32_t a_left = a_steps, b_left = b_steps;
  // scalar offsets from one stage to the next, and from the last stage of a
  // K block to the first of the next
  const uint32_t a_adv = kBK8x, a_adv_wrap = (uint32_t)(kBK8x + p.a.slice - p.a.kslice);
  const uint32_t b_adv = (uint32_t)(kBK8x * p.b.ld);
  const uint32_t b_adv_wrap = (uint32_t)(b_adv + p.b.slice - (int64_t)p.b.kslice * p.b.ld);
  uint32_t a_so = 0, b_so = 0;
  struct StageSrc {
    i32x4 ra, rb;
    uint32_t sa, sb;
  };
  // The next stage: the descriptors (empty past the last step, so no memory
  // is touched) and the stage's byte offsets.
  auto next_src = [&](bool live) __attribute__((always_inline)) {
    StageSrc d;
    d.ra = a_desc;
    d.rb = b_desc;
    if (!live) d.ra[2] = d.rb[2] = 0;
    d.sa = a_so;
    d.sb = b_so;
    const bool a_wrap = --a_left == 0;
    a_so += a_wrap ? a_adv_wrap : a_adv;
    a_left = a_wrap ? a_steps : a_left;
    const bool b_wrap = --b_left == 0;
    b_so += b_wrap ? b_adv_wrap : b_adv;
    b_left = b_wrap ? b_steps : b_left;
    return d;
  };
  // A wave's loads of one operand in one stage form a run sharing one M0
  // write (LDS rows 1 KiB apart, 1024 i in the instruction offset).
  auto load_one = [&](const StageSrc& d, char* sA, char* sB, int i) __attribute__((always_inline)) {
    if (i == 0) lds_dma16_first(d.ra, a_voff[0], d.sa, sA + wave * T::NA * 1024);
    else if (i == 1) lds_dma16_next<1024>(d.ra, a_voff[1], d.sa);
    else if (i == 2) lds_dma16_next<2048>(d.ra, a_voff[2], d.sa);
    else if (i == 3) lds_dma16_next<3072>(d.ra, a_voff[3], d.sa);
    else if (i == 4) lds_dma16_first(d.rb, b_voff[0], d.sb, sB + wave * T::NB * 1024);
    else if (i == 5) lds_dma16_next<1024>(d.rb, b_voff[1], d.sb);
    else if (i == 6) lds_dma16_next<2048>(d.rb, b_voff[2], d.sb);
    else lds_dma16_next<3072>(d.rb, b_voff[3], d.sb);
  };
  static_assert(T::NA == 4 && T::NB == 4, "load runs of 4 per operand and stage");

  i32x8 fa[2];                        // A tile mt in fa[mt % 2]
  i32x8 F0, F1, F2, F3, S0, S1;       // B fragments: four current, two spare
  auto read_a = [&](const char* sA, int mt, i32x8& f) __attribute__((always_inline)) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const i32x4v v = *(const lds_i32x4*)(sA + a_rd[h] + mt * 16 * kBK8x);
#pragma unroll
      for (int q = 0; q < 4; ++q) f[4 * h + q] = v[q];
    }
  };
  auto read_b = [&](const char* sB, int nt, i32x8& f) __attribute__((always_inline)) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const i32x2 v = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2*)(sB + b_rd[nt][r]));
      f[2 * r] = v[0];
      f[2 * r + 1] = v[1];
    }
  };

  f32x4 acc[T::TM][T::TN];
#pragma unroll
  for (int i = 0; i < T::TM; ++i)
#pragma unroll
    for (int j = 0; j < T::TN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[i][j][v] = 0.f;
  auto mfma = [&](int mt, int nt, const i32x8& b) __attribute__((always_inline)) {
    acc[mt][nt] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(b, fa[mt & 1], acc[mt][nt], 0, 0,
                                                                  0, 0, 0, 0);
  };
  auto barrier = [&](auto VM) __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(decltype(VM)::value, 0));
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  // One step on stage t (A buffer sa, B buffer sb), with the current B
  // fragments in (b0 .. b3) and the spares (s0, s1); stage t + 1 is in
  // (na, nb); the loads of stage t + 2 go to (la, lb) with descriptors d.
  // On return the next step's B fragments are (s0, s1, b2, b3) and its A
  // tile 0 is in fa[0].
  auto step = [&](const char* sa, const char* na, const char* nb, char* la, char* lb,
                  const StageSrc& d, i32x8& b0, i32x8& b1, i32x8& b2, i32x8& b3, i32x8& s0,
                  i32x8& s1) __attribute__((always_inline)) {
    // row 0 (nt 0..3), A tile 1 behind it
    mfma(0, 0, b0);
    read_a(sa, 1, fa[1]);
    __builtin_amdgcn_sched_barrier(0);
    mfma(0, 1, b1);
    mfma(0, 2, b2);
    mfma(0, 3, b3);
    __builtin_amdgcn_sched_barrier(0);
    barrier(std::integral_constant<int, 63>{});                          // X
    // rows 1-5; the loads of stage t + 2 behind rows 1-2
#pragma unroll
    for (int mt = 1; mt <= T::ROW_Y; ++mt) {
#pragma unroll
      for (int j = 0; j < T::TN; ++j) {
        const int nt = (mt & 1) ? T::TN - 1 - j : j;
        mfma(mt, nt, nt == 0 ? b0 : nt == 1 ? b1 : nt == 2 ? b2 : b3);
        if (j == 0) read_a(sa, mt + 1, fa[(mt + 1) & 1]);
        if (mt <= 2) load_one(d, la, lb, 4 * (mt - 1) + j);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    barrier(std::integral_constant<int, T::NL>{});                       // Y
    // row 6 (nt 0..3): A tile 7 and the next step's B tiles 0, 1 (spares)
    mfma(6, 0, b0);
    read_a(sa, 7, fa[1]);
    __builtin_amdgcn_sched_barrier(0);
    mfma(6, 1, b1);
    read_b(nb, 0, s0);
    __builtin_amdgcn_sched_barrier(0);
    mfma(6, 2, b2);
    read_b(nb, 1, s1);
    __builtin_amdgcn_sched_barrier(0);
    mfma(6, 3, b3);
    __builtin_amdgcn_sched_barrier(0);
    // row 7 (nt 3..0): the next A tile 0 goes to fa[0] first (LDS reads
    // complete in order, and the next step's first MFMA needs it); the next
    // B tiles 3, 2 replace the current ones after their last MFMA
    mfma(7, 3, b3);
    read_a(na, 0, fa[0]);
    read_b(nb, 3, b3);
    __builtin_amdgcn_sched_barrier(0);
    mfma(7, 2, b2);
    read_b(nb, 2, b2);
    __builtin_amdgcn_sched_barrier(0);
    mfma(7, 1, b1);
    mfma(7, 0, b0);
    __builtin_amdgcn_sched_barrier(0);
  };

  // Prologue: stages 0 and 1 in flight; then stage 0's B fragments and A
  // tile 0.
  {
    const StageSrc d0 = next_src(0 < ksteps);
#pragma unroll
    for (int i = 0; i < T::NL; ++i) load_one(d0, smA[0], smB[0], i);
    const StageSrc d1 = next_src(1 < ksteps);
#pragma unroll
    for (int i = 0; i < T::NL; ++i) load_one(d1, smA[1], smB[1], i);
  }
  barrier(std::integral_constant<int, T::NL>{});
  read_b(smB[0], 0, F0);
  read_b(smB[0], 1, F1);
  read_b(smB[0], 2, F2);
  read_b(smB[0], 3, F3);
  read_a(smA[0], 0, fa[0]);

  // Step t (phase ph = t mod 6): A buffer ph % 3, B buffer ph % 2; the loads
  // of stage t + 2 go to A buffer (ph + 2) % 3 and B buffer ph % 2.
  auto phase_step = [&](auto PH, int32_t t, bool all_live) __attribute__((always_inline)) {
    constexpr int ph = decltype(PH)::value;
    const StageSrc d = next_src(all_live || t + 2 < ksteps);
    if constexpr (ph % 2 == 0)
      step(smA[ph % 3], smA[(ph + 1) % 3], smB[(ph + 1) % 2], smA[(ph + 2) % 3], smB[ph % 2], d,
           F0, F1, F2, F3, S0, S1);
    else
      step(smA[ph % 3], smA[(ph + 1) % 3], smB[(ph + 1) % 2], smA[(ph + 2) % 3], smB[ph % 2], d,
           S0, S1, F2, F3, F0, F1);
  };
  // Groups of 6 steps whose loads (stages up to t + 7) all exist, then the
  // remaining steps (at most 7) in groups of 6 with each step behind a
  // (uniform) bound check.
  int32_t t = 0;
  for (; t + 8 <= ksteps; t += 6) {
    phase_step(std::integral_constant<int, 0>{}, t, true);
    phase_step(std::integral_constant<int, 1>{}, t + 1, true);
    phase_step(std::integral_constant<int, 2>{}, t + 2, true);
    phase_step(std::integral_constant<int, 3>{}, t + 3, true);
    phase_step(std::integral_constant<int, 4>{}, t + 4, true);
    phase_step(std::integral_constant<int, 5>{}, t + 5, true);
  }
#define CCL_FP8P_PHASE(k) \
  if (t + k < ksteps) phase_step(std::integral_constant<int, k>{}, t + k, false)
  for (; t < ksteps; t += 6) {
    CCL_FP8P_PHASE(0); CCL_FP8P_PHASE(1); CCL_FP8P_PHASE(2);
    CCL_FP8P_PHASE(3); CCL_FP8P_PHASE(4); CCL_FP8P_PHASE(5);
  }
#undef CCL_FP8P_PHASE

  static_assert((BM / 2) * BN * 2 <= T::NSA * T::A_BYTES && (BM / 2) * BN * 2 <= T::NSB * T::B_BYTES,
                "each half of the bf16 C tile fits in one operand's stage buffers");
  // The lane index, made opaque here so that the epilogue's addresses are
  // computed after the K loop instead of being hoisted before it (where
  // they would stay live through the loop and spill).
  int ln = lane;
  asm volatile("" : "+v"(ln));
  // Non-temporal C stores: at the power limit the fp8 GEMMs ran 1-4 % faster
  // with them, at a 1 % higher clock (same box, alternating).
  if (p.epi == 0 && !p.c_f32 && !p.ws)
    store_tile_staged<BM, BN, T::NW, T::TM, T::TN, T::WM, T::WN, true>(
        p, acc, &smA[0][0], &smB[0][0], pr, pc, ti, tj, wm, wn, wave, ln);
  else
    store_tile<BM, BN, 16, T::TM, T::TN, T::WM, T::WN>(p, acc, pr, pc, ti, tj, split, wm, wn, ln);
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

// Split-K workspace of ccl_gemm_splitk_noalloc: the fp32 partial tiles
// live in this array instead of caller memory. Each GPU holds its own copy
// (allocated when the library's code object is loaded on it). Nothing in it
// needs clearing: every K range writes its whole partial tile before the
// reduce launch reads it. Calls that overlap on one GPU share it and race.
static __device__ __align__(256) float scratch[kScratchBytes / sizeof(float)];

namespace {
constexpr int kScratchDevices = 64;
std::once_flag g_scratch_once[kScratchDevices];
float* g_scratch_ptr[kScratchDevices];
hipError_t g_scratch_err[kScratchDevices];
}  // namespace

// Host code must not pass `scratch` itself to a kernel (on the host the name
// is only a stand-in): the device address comes from the runtime, once per
// device, with that device current.
hipError_t scratch_workspace(float** ws) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
  std::call_once(g_scratch_once[dev], [dev] {
    void* ptr = nullptr;
    g_scratch_err[dev] = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    g_scratch_ptr[dev] = static_cast<float*>(ptr);
  });
  if (g_scratch_err[dev] != hipSuccess) return g_scratch_err[dev];
  if (g_scratch_ptr[dev] == nullptr) return hipErrorInvalidSymbol;
  *ws = g_scratch_ptr[dev];
  return hipSuccess;
}

// Second launch of a split-K GEMM: sum the partials of every tile into C.
static hipError_t launch_splitk_reduce(const Plan& p, GemmParams gp, hipStream_t stream) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  gp.map = tile_map(p, 1);
  const dim3 grid((unsigned)splitk_reduce_workgroups(p));
  const GemmConfig& g = p.gemm;
  // The partials are in the fragment order of the kernel that wrote them:
  // 16x16 MFMA tiles for bf16, 32x32 for fp8.
  const int md = p.ab_type == DT_FP8_E4M3 ? 32 : 16;
#define CCL_REDUCE(BM_, BN_, WGN_, MD_) \
  hipLaunchKernelGGL((splitk_reduce_kernel<BM_, BN_, WGN_, MD_>), grid, dim3(256), 0, stream, gp)
#define CCL_REDUCE_MD(BM_, BN_, WGN_) \
  do { if (md == 16) CCL_REDUCE(BM_, BN_, WGN_, 16); else CCL_REDUCE(BM_, BN_, WGN_, 32); } while (0)
  if (g.tile_m == 256 && g.tile_n == 256 && g.waves == 8) CCL_REDUCE_MD(256, 256, 4);
  else if (g.tile_m == 256 && g.tile_n == 128 && g.waves == 8) CCL_REDUCE_MD(256, 128, 4);
  else if (g.tile_m == 128 && g.tile_n == 256 && g.waves == 8) CCL_REDUCE_MD(128, 256, 4);
  else if (g.tile_m == 128 && g.tile_n == 128 && g.waves == 8) CCL_REDUCE_MD(128, 128, 4);
  else if (g.tile_m == 256 && g.tile_n == 256) CCL_REDUCE_MD(256, 256, 2);
  else if (g.tile_m == 256 && g.tile_n == 128) CCL_REDUCE_MD(256, 128, 2);
  else if (g.tile_m == 128 && g.tile_n == 256) CCL_REDUCE_MD(128, 256, 2);
  else if (g.tile_m == 128 && g.tile_n == 128) CCL_REDUCE_MD(128, 128, 2);
  else return hipErrorInvalidValue;
#undef CCL_REDUCE_MD
#undef CCL_REDUCE
  return hipGetLastError();
}

hipError_t launch_gemm(const Plan& p, const void* A, const void* B, void* C,
                       const OperandAddr& a, const OperandAddr& b, const OperandAddr& c,
                       bool remap, float alpha, float beta, int splits, float* ws,
                       hipStream_t stream, uint64_t* timeline) {
  const GemmConfig& g = p.gemm;
  GemmParams gp;
  gp.timeline = timeline;
  gp.A = static_cast<const uint16_t*>(A);
  gp.B = static_cast<const uint16_t*>(B);
  gp.C = C;
  gp.c_f32 = p.c_type == DT_FP32 ? 1 : 0;
  gp.a = a;
  gp.b = b;
  gp.c = c;
  if (splits < 1 || (splits > 1 && (!remap || !ws))) return hipErrorInvalidValue;
  splits = effective_splits(p, splits);      // every K range non-empty
  gp.map = tile_map(p, splits);
  const bool fp8 = p.ab_type == DT_FP8_E4M3;
  if (timeline && (fp8 || splits > 1)) return hipErrorInvalidValue;   // bf16 kernel only
  gp.ksteps = (int32_t)(p.K / (fp8 ? kBK8 : kBK));
  gp.ksteps_per_split = (gp.ksteps + splits - 1) / splits;
  // Rounds path of the bf16 kernel: each operand's K blocks are a multiple
  // of 4 steps (or it has one block), and every split starts 4-aligned.
  {
    const auto aligned = [&](const OperandAddr& o) {
      return (int64_t)o.kslice == p.K || (o.kslice / kBK) % 4 == 0;
    };
    gp.round_fast = (!fp8 && kStagesBf16 == 4 && aligned(a) && aligned(b) &&
                     (splits == 1 || gp.ksteps_per_split % 4 == 0)) ? 1 : 0;
  }
  gp.splits_total = splits;
  gp.ws = splits > 1 ? ws : nullptr;
  gp.remap = remap ? 1 : 0;
  gp.grid_r = p.Gr;
  gp.alpha = alpha;
  gp.beta = beta;
  gp.epi = beta != 0.f ? 2 : (alpha != 1.f ? 1 : 0);
  const unsigned wgs = remap ? (unsigned)(8 * (int64_t)gp.map.tiles_per_xcd)
                             : (unsigned)(g.tiles_m * g.tiles_n * p.G);
  dim3 grid(wgs);
  const int waves = g.waves;
  // fp8 on 256x256 tiles with 8 waves: the 16x16x128 kernel, where every
  // K block is a multiple of its 128-wide step (no split-K). Other fp8
  // plans run the 32x32x64 kernel.
  if (fp8 && splits == 1 && waves == 8 && g.tile_m == 256 && g.tile_n == 256 &&
      a.kslice % kBK8x == 0 && b.kslice % kBK8x == 0) {
    gp.ksteps = (int32_t)(p.K / kBK8x);
    gp.ksteps_per_split = gp.ksteps;
    // the pipelined kernel's descriptors span the tile's rows of A and
    // columns of B over all K blocks
    const int64_t lim = ((int64_t)1 << 31) - 4096;
    const bool fits = (p.K / a.kslice - 1) * a.slice + 256 * (int64_t)a.ld < lim &&
                      (p.K / b.kslice - 1) * b.slice + (int64_t)b.kslice * b.ld + 256 < lim;
    if (g.fp8_pipe && fits) {
      hipLaunchKernelGGL(gemm_fp8p_kernel, grid, dim3(TileFp8P::THREADS), 0, stream, gp);
      return hipGetLastError();
    }
    hipLaunchKernelGGL((gemm_fp8x_kernel<256, 256, 4>), grid, dim3(Tile8x<256, 256, 4>::THREADS), 0,
                       stream, gp);
    return hipGetLastError();
  }
  if (fp8) {
#define CCL_LAUNCH8(BM_, BN_, WGN_)                                                    \
  hipLaunchKernelGGL((gemm_fp8_kernel<BM_, BN_, WGN_>), grid, dim3(Tile8<BM_, BN_, WGN_>::THREADS), \
                     0, stream, gp)
    if (g.tile_m == 256 && g.tile_n == 256 && waves == 8)
      CCL_LAUNCH8(256, 256, 4);
    else if (g.tile_m == 256 && g.tile_n == 256)
      CCL_LAUNCH8(256, 256, 2);
    else if (g.tile_m == 256 && g.tile_n == 128)
      CCL_LAUNCH8(256, 128, 2);
    else if (g.tile_m == 128 && g.tile_n == 256)
      CCL_LAUNCH8(128, 256, 2);
    else if (g.tile_m == 128 && g.tile_n == 128)
      CCL_LAUNCH8(128, 128, 2);
    else
      return hipErrorInvalidValue;
#undef CCL_LAUNCH8
    return splits > 1 ? launch_splitk_reduce(p, gp, stream) : hipGetLastError();
  }
  // 64-K stages (plan's choice for the bf16 tiles below 256x256): both K
  // blocks a multiple of 64, the 4-step rounds' extents (255 rows of A or
  // B) within 32-bit offsets, and with split-K only where the K ranges are
  // the 32-K ranges (each range an even number of 32-K steps), so the
  // workspace and the reduce are unchanged.
  {
    const int64_t lim = ((int64_t)1 << 31) - 4096;
    const int32_t ks64 = (int32_t)(p.K / kBK64);
    const int32_t per64 = (ks64 + splits - 1) / splits;
    const bool k64 = g.stage_k == 64 && !fp8 && waves == 8 &&
                     !(g.tile_m == 256 && g.tile_n == 256) && a.kslice % kBK64 == 0 &&
                     b.kslice % kBK64 == 0 && 255 * (int64_t)a.ld * 2 + 512 < lim &&
                     255 * (int64_t)b.ld * 2 + 512 < lim && 2 * per64 == gp.ksteps_per_split;
    if (k64) {
      const auto aligned64 = [&](const OperandAddr& o) {
        return (int64_t)o.kslice == p.K || (o.kslice / kBK64) % 4 == 0;
      };
      gp.ksteps = ks64;
      gp.ksteps_per_split = per64;
      gp.round_fast = aligned64(a) && aligned64(b) && (splits == 1 || per64 % 4 == 0) ? 1 : 0;
#define CCL_LAUNCH64(BM_, BN_)                                                                \
  hipLaunchKernelGGL((gemm_k64_kernel<BM_, BN_>), grid, dim3(Tile64<BM_, BN_>::THREADS), 0, stream, gp)
      if (g.tile_m == 256 && g.tile_n == 128) CCL_LAUNCH64(256, 128);
      else if (g.tile_m == 128 && g.tile_n == 256) CCL_LAUNCH64(128, 256);
      else if (g.tile_m == 128 && g.tile_n == 128) CCL_LAUNCH64(128, 128);
      else return hipErrorInvalidValue;
#undef CCL_LAUNCH64
      return splits > 1 ? launch_splitk_reduce(p, gp, stream) : hipGetLastError();
    }
  }
  // The 64-K-pair kernel's A descriptor spans the tile's 256 rows over all
  // K blocks of A.
  if (g.a_pairs && !fp8 && splits == 1 && waves == 8 && g.tile_m == 256 && g.tile_n == 256 &&
      a.kslice % 64 == 0 &&
      (p.K / a.kslice - 1) * a.slice * 2 + 256 * (int64_t)a.ld * 2 + 4096 < ((int64_t)1 << 31)) {
    hipLaunchKernelGGL(gemm_a2_kernel, grid, dim3(TileA2::THREADS), 0, stream, gp);
    return hipGetLastError();
  }
#define CCL_LAUNCH(BM_, BN_, WGN_)                                                     \
  hipLaunchKernelGGL((gemm_kernel<BM_, BN_, WGN_>), grid, dim3(Tile<BM_, BN_, WGN_>::THREADS), 0, \
                     stream, gp)
  if (g.tile_m == 256 && g.tile_n == 256 && waves == 8)
    CCL_LAUNCH(256, 256, 4);
  else if (g.tile_m == 256 && g.tile_n == 128 && waves == 8)
    CCL_LAUNCH(256, 128, 4);
  else if (g.tile_m == 128 && g.tile_n == 256 && waves == 8)
    CCL_LAUNCH(128, 256, 4);
  else if (g.tile_m == 128 && g.tile_n == 128 && waves == 8)
    CCL_LAUNCH(128, 128, 4);
  else if (g.tile_m == 256 && g.tile_n == 256)
    CCL_LAUNCH(256, 256, 2);
  else if (g.tile_m == 256 && g.tile_n == 128)
    CCL_LAUNCH(256, 128, 2);
  else if (g.tile_m == 128 && g.tile_n == 256)
    CCL_LAUNCH(128, 256, 2);
  else if (g.tile_m == 128 && g.tile_n == 128)
    CCL_LAUNCH(128, 128, 2);
  else
    return hipErrorInvalidValue;
#undef CCL_LAUNCH
  return splits > 1 ? launch_splitk_reduce(p, gp, stream) : hipGetLastError();
}

hipError_t launch_dispatch_probe(const Plan& p, int32_t* out, hipStream_t stream) {
  hipLaunchKernelGGL(dispatch_probe_kernel, dim3((unsigned)p.gemm.workgroups), dim3(64), 0, stream,
                     tile_map(p), (int32_t)p.gemm.tiles_m, (int32_t)p.gemm.tiles_n, out);
  return hipGetLastError();
}

}  // namespace ccl
