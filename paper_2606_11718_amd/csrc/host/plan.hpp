// Host-side plan of a CCL GEMM: validation, per-operand CCL layouts, tile
// ownership, the workgroup -> XCD -> tile map of the GEMM launch, and the
// remote-byte model. Plain C++17, no HIP dependency.
#pragma once

#include <cstdint>
#include <string>

#include "tile_map.hpp"

namespace ccl {

constexpr int kModelTile = 128;   // output tile of the traffic model (Sec. IV-A)
constexpr int kNumXcd = 8;        // MI355X: 8 XCDs, workgroups dispatched round-robin
constexpr int kMaxChiplets = 64;
constexpr int kGemmBK = 32;       // K extent of one GEMM main-loop step (bf16)
constexpr int kGemmBK8 = 64;      // the same for fp8 operands
constexpr int kMaxSplits = 16;    // split-K ranges per tile

enum Op { OP_A = 0, OP_B = 1, OP_C = 2 };
// Element types (Fig. 7 sweeps the data type): A and B share one type.
enum DType { DT_BF16 = 0, DT_FP8_E4M3 = 1, DT_FP32 = 2 };
inline int dtype_bytes(DType t) { return t == DT_FP8_E4M3 ? 1 : (t == DT_FP32 ? 4 : 2); }
enum Placement { PLACE_RR = 0, PLACE_COARSE = 1, PLACE_CCL = 2 };

struct Layout {
  int64_t rows = 0, cols = 0;
  int64_t grid_r = 0, grid_c = 0;
  int64_t block_rows = 0, block_cols = 0;
  int64_t strip_bytes = 0, strip_stride_bytes = 0, total_bytes = 0;
  int64_t elem_bytes = 2;

  // Byte offset of logical element (r, c) (Sec. III-B, block form of Eq. 3).
  int64_t offset(int64_t r, int64_t c) const {
    int64_t b = (r / block_rows) * grid_c + (c / block_cols);
    return b * strip_stride_bytes + ((r % block_rows) * block_cols + (c % block_cols)) * elem_bytes;
  }
};

// Kernel-level tiling chosen for a plan (kernel tiles nest inside partitions).
struct GemmConfig {
  int tile_m = 0, tile_n = 0;       // kernel output tile
  int64_t tiles_m = 0, tiles_n = 0; // kernel tiles per partition
  int xcd_per_chiplet = 0;          // 8 / G
  int64_t tiles_per_xcd = 0;        // ceil(tiles per partition / xcd_per_chiplet)
  int64_t workgroups = 0;           // 8 * tiles_per_xcd
  int group_m = 0;                  // raster group height (tiles) inside a partition
  int waves = 4;                    // waves per workgroup (4 or 8)
  int stage_k = 32;                 // bf16: K extent of one LDS stage (32 or 64)
  bool a_pairs = false;             // bf16 256x256: A staged in 64-K pairs (whole lines)
  bool fp8_pipe = false;            // fp8 256x256: fragment reads pipelined across steps
  bool supported = false;           // whether ccl_gemm can run this plan
  std::string why_unsupported;
};

struct Traffic {
  uint64_t accessed[3] = {0, 0, 0};
  uint64_t remote[3] = {0, 0, 0};
  uint64_t floor_bytes = 0;
  uint64_t footprint[3] = {0, 0, 0};
  uint64_t remote_per_chiplet[kMaxChiplets] = {};
  int chiplets = 0;
};

struct Plan {
  int64_t M = 0, N = 0, K = 0;
  int G = 0, Gr = 0, Gc = 0;
  int64_t page = 0;
  DType ab_type = DT_BF16, c_type = DT_BF16;
  Layout lay[3];
  GemmConfig gemm;

  int64_t part_rows() const { return M / Gr; }
  int64_t part_cols() const { return N / Gc; }
  // Chiplet owning the 128x128 model tile (ti, tj).
  int owner(int64_t ti, int64_t tj) const {
    return static_cast<int>((ti * kModelTile / part_rows()) * Gc + (tj * kModelTile / part_cols()));
  }
};

enum class Status { OK = 0, INVALID_ARG = 1, UNALIGNED = 2, UNSUPPORTED = 3, MISALIGNED = 4, HIP = 5 };

// Build a plan. grid_rows == 0 chooses the grid. On error returns the status
// and fills `err` with a message. ab: type of A and B (bf16, fp8 E4M3, or
// fp32 for layouts and traffic models only); c: type of C (bf16 or fp32).
Status make_plan(int64_t M, int64_t N, int64_t K, int chiplets, int grid_rows, int64_t page,
                 DType ab, DType c, Plan* out, std::string* err);

// Whether a Gr x (G/Gr) grid gives tile-aligned partitions.
bool grid_aligned(int64_t M, int64_t N, int64_t K, int G, int Gr);

// Remote bytes of CCL (the floor):
// M*N*K*[e_A*(Gc-1)/(Gc*128) + e_B*(Gr-1)/(Gr*128)].
uint64_t floor_bytes(int64_t M, int64_t N, int64_t K, int Gr, int Gc, int ea, int eb);

// Traffic flags: bit 0 A stored transposed, bit 1 B stored transposed,
// bit 2 C is read as well as written (alpha A B + beta C with beta != 0).
constexpr int kTrafficCRead = 4;

// The remote-byte model under one placement.
Traffic remote_bytes(const Plan& p, Placement pl, int flags);

// Parameters of the workgroup -> tile map of the GEMM launch (splits > 1:
// the split-K launch).
TileMap tile_map(const Plan& p, int splits = 1);

// GEMM main-loop steps over K (32 bf16 or 64 fp8 elements each).
int64_t gemm_ksteps(const Plan& p);

// Split-K: the split count that fills an XCD's CUs for this plan (1 when
// the partition already has enough tiles); the number of non-empty K ranges
// when the K steps are cut into ranges of ceil(steps / splits); and the fp32
// workspace that needs (tiles x ranges x tile elements x 4 bytes, 0 for one
// range).
int recommended_splits(const Plan& p);
int effective_splits(const Plan& p, int splits);
int64_t splitk_workspace_bytes(const Plan& p, int splits);
// Workgroups of the split-K GEMM launch and of its reduce launch (one per
// 256 x float4 chunk of every tile).
int64_t splitk_workgroups(const Plan& p, int splits);
int64_t splitk_reduce_workgroups(const Plan& p);

// Workgroup -> (xcd, kernel tile) of the GEMM launch; tile = (-1, -1) if idle.
void tile_of_wg(const Plan& p, int64_t wg, int* xcd, int64_t* tile_m, int64_t* tile_n);

}  // namespace ccl
