// Host-side plan of a CCL GEMM (see plan.hpp).
//
// Remote-byte model (Sec. IV-A "Metrics"; no cache): every 128x128 output
// tile runs on its owner chiplet, reads its whole A row panel and B column
// panel and writes its C tile; an element access is remote when the page
// holding the element sits on another chiplet. The model here walks, for
// each panel, the byte intervals the panel occupies in the stored tensor
// and splits every interval at page boundaries, so the per-chiplet counts
// come from interval lengths rather than from element enumeration.
#include "plan.hpp"

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

namespace ccl {

namespace {

bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

Layout make_layout(int64_t rows, int64_t cols, int Gr, int Gc, int64_t page, int e) {
  Layout l;
  l.elem_bytes = e;
  l.rows = rows;
  l.cols = cols;
  l.grid_r = Gr;
  l.grid_c = Gc;
  l.block_rows = rows / Gr;
  l.block_cols = cols / Gc;
  l.strip_bytes = l.block_rows * l.block_cols * e;
  l.strip_stride_bytes = (l.strip_bytes + page - 1) / page * page;
  l.total_bytes = l.strip_stride_bytes * Gr * Gc;
  return l;
}

// Extra bytes of the shared operands that their non-owning sharers need,
// scaled by G to stay an integer: e_A*M*K*(Gc-1)*Gr + e_B*K*N*(Gr-1)*Gc.
unsigned __int128 replicated_times_g(int64_t M, int64_t N, int64_t K, int Gr, int Gc, int ea, int eb) {
  unsigned __int128 a = (unsigned __int128)M * K * (Gc - 1) * Gr * ea;
  unsigned __int128 b = (unsigned __int128)K * N * (Gr - 1) * Gc * eb;
  return a + b;
}

// Panels (distinct tile rows plus distinct tile columns) that the waves of
// 32 co-resident tiles touch, summed over the XCDs of one chiplet, when each
// XCD walks its range of the partition's tiles in groups of gm tile rows,
// each group column by column (the order of map_tile in tile_map.hpp).
int64_t panels_touched(const GemmConfig& g, int gm) {
  const int64_t tiles = g.tiles_m * g.tiles_n;
  const int64_t h0 = std::min<int64_t>(gm, g.tiles_m);
  const int64_t per_group = h0 * g.tiles_n;
  int64_t total = 0;
  std::vector<char> row_seen(g.tiles_m), col_seen(g.tiles_n);
  for (int64_t sub = 0; sub < g.xcd_per_chiplet; ++sub) {
    for (int64_t w0 = 0; w0 < g.tiles_per_xcd; w0 += 32) {
      std::fill(row_seen.begin(), row_seen.end(), 0);
      std::fill(col_seen.begin(), col_seen.end(), 0);
      for (int64_t slot = w0; slot < std::min<int64_t>(w0 + 32, g.tiles_per_xcd); ++slot) {
        const int64_t t = sub * g.tiles_per_xcd + slot;
        if (t >= tiles) break;
        const int64_t first = (t / per_group) * h0;
        const int64_t h = std::min<int64_t>(h0, g.tiles_m - first);
        const int64_t w = t - (t / per_group) * per_group;
        const int64_t ti = first + w % h, tj = w / h;
        total += (row_seen[ti] ? 0 : 1) + (col_seen[tj] ? 0 : 1);
        row_seen[ti] = col_seen[tj] = 1;
      }
    }
  }
  return total;
}

void choose_gemm_config(Plan* p) {
  GemmConfig& g = p->gemm;
  g = GemmConfig();
  const int64_t pr = p->part_rows(), pc = p->part_cols();
  if (kNumXcd % p->G != 0) {
    g.why_unsupported = "chiplets must divide the 8 XCDs";
    return;
  }
  if (p->ab_type == DT_FP32) {
    g.why_unsupported = "the GEMM kernels take bf16 or fp8 A and B (fp32 plans serve layouts and traffic models)";
    return;
  }
  const int64_t bk = p->ab_type == DT_FP8_E4M3 ? kGemmBK8 : kGemmBK;
  if ((p->K / p->Gc) % bk != 0 || (p->K / p->Gr) % bk != 0) {
    g.why_unsupported = p->ab_type == DT_FP8_E4M3
                            ? "fp8: K / grid_cols and K / grid_rows must be multiples of 64"
                            : "K / grid_cols and K / grid_rows must be multiples of 32";
    return;
  }
  g.xcd_per_chiplet = kNumXcd / p->G;
  // Candidate kernel tiles, largest first; estimated time = waves of 32
  // workgroups per XCD times the tile's work over a per-tile efficiency.
  struct Cand { int tm, tn; double eff; };
  const Cand cands[] = {{256, 256, 1.0}, {256, 128, 0.85}, {128, 256, 0.85}, {128, 128, 0.7}};
  double best = 0;
  int btm = 0, btn = 0;
  const char* forced = std::getenv("CCL_GEMM_TILE");
  int ftm = 0, ftn = 0;
  if (forced && std::sscanf(forced, "%dx%d", &ftm, &ftn) != 2) ftm = ftn = 0;
  for (const Cand& c : cands) {
    if (pr % c.tm || pc % c.tn) continue;
    if (ftm && (c.tm != ftm || c.tn != ftn)) continue;
    int64_t tiles = (pr / c.tm) * (pc / c.tn);
    int64_t per_xcd = (tiles + g.xcd_per_chiplet - 1) / g.xcd_per_chiplet;
    int64_t waves = (per_xcd + 31) / 32;
    double t = (double)waves * c.tm * c.tn / c.eff;
    if (btm == 0 || t < best) {
      best = t;
      btm = c.tm;
      btn = c.tn;
    }
  }
  if (btm == 0) {
    g.why_unsupported = "no kernel tile fits the partitions (or CCL_GEMM_TILE does not)";
    return;
  }
  g.tile_m = btm;
  g.tile_n = btn;
  g.tiles_m = pr / btm;
  g.tiles_n = pc / btn;
  g.tiles_per_xcd = (g.tiles_m * g.tiles_n + g.xcd_per_chiplet - 1) / g.xcd_per_chiplet;
  g.workgroups = g.tiles_per_xcd * kNumXcd;
  // Raster group height. An XCD runs 32 tiles at once (one workgroup per CU);
  // 4 tile rows x 8 tile columns make them share 12 A row panels and B
  // column panels, which the XCD's L2 serves while they step through K
  // together. Where a group is not a whole number of such waves, some waves
  // straddle two groups and touch more panels. So the height is the one of
  // 4 and 8 whose waves touch the fewest panels in total (4 on a tie: on
  // 8192x8192x28672 both give 12 per wave and 4 measured 1.5 % faster).
  // Measured on 8192x28672x8192 (28 tile columns, 8 rows chosen): 9 % less
  // L2-miss traffic than 4 rows, 1 % faster.
  int gm = panels_touched(g, 8) < panels_touched(g, 4) ? 8 : 4;
  if (const char* e = std::getenv("CCL_GEMM_GROUP_M")) gm = std::max(1, std::atoi(e));
  g.group_m = (int)std::min<int64_t>(gm, g.tiles_m);
  // Waves per workgroup: 8 (two per SIMD) for every bf16 tile and for fp8
  // 256x256 tiles, 4 for the other fp8 tiles. On the Qwen3 shapes the 8-wave
  // forms of the 256x128 and 128x128 tiles measured 0-10 % faster than 4.
  // CCL_GEMM_WAVES=4 selects the 4-wave form.
  const bool eight_ok = (btm == 256 && btn == 256) || p->ab_type == DT_BF16;
  g.waves = eight_ok ? 8 : 4;
  if (const char* e = std::getenv("CCL_GEMM_WAVES"))
    g.waves = (std::atoi(e) == 8 && eight_ok) ? 8 : 4;
  // LDS stage depth in K (bf16). A stage of 32 K holds 64-byte A rows, half
  // a 128-byte line, and a CU streams such half lines from L2 at 36-47
  // B/clk when most CUs load, against 57-64 B/clk for whole lines
  // (direct-to-LDS loads of L2-resident data). The tiles below 256x256 need
  // 48-64 B/clk per CU at the matrix cores' rate, so they take 64-K stages
  // (whole-line A rows), where both K blocks allow it. 256x256 keeps 32:
  // two 64-K stages would leave one step of load lookahead.
  // CCL_GEMM_STAGE_K=32 selects the 32-K stages everywhere.
  g.stage_k = (p->ab_type == DT_BF16 && g.waves == 8 && !(btm == 256 && btn == 256) &&
               (p->K / p->Gc) % 64 == 0 && (p->K / p->Gr) % 64 == 0) ? 64 : 32;
  if (const char* e = std::getenv("CCL_GEMM_STAGE_K"))
    if (std::atoi(e) == 32) g.stage_k = 32;
  // 256x256 keeps 32-K steps for B and the MFMA schedule but stages A in
  // 64-K pairs of steps: whole 128-byte lines per A load, and loads four
  // steps ahead in a ring of three pair buffers. Same box, alternating:
  // 8192x28672x8192 1416-1423 -> 1484-1492 TFLOP/s, 8192x8192x28672
  // 1433-1437 -> 1504-1508, at the same 1400 W. Needs A's K blocks in
  // whole pairs. CCL_GEMM_A_PAIRS=0 selects the 32-K A stages.
  g.a_pairs = p->ab_type == DT_BF16 && g.waves == 8 && btm == 256 && btn == 256 &&
              (p->K / p->Gc) % 64 == 0;
  if (const char* e = std::getenv("CCL_GEMM_A_PAIRS"))
    if (std::atoi(e) == 0) g.a_pairs = false;
  // fp8 256x256 (16x16x128 kernel): three A and two B stage buffers, two
  // barriers per step, and the next step's fragments read behind the last
  // rows of MFMAs (gemm_fp8p_kernel). CCL_GEMM_FP8_PIPE=0 selects the
  // two-stage kernel that reads them after each step's barrier.
  g.fp8_pipe = p->ab_type == DT_FP8_E4M3 && g.waves == 8 && btm == 256 && btn == 256;
  if (const char* e = std::getenv("CCL_GEMM_FP8_PIPE"))
    if (std::atoi(e) == 0) g.fp8_pipe = false;
  if (g.workgroups > 0x7fffffff) {
    g.why_unsupported = "launch too large";
    return;
  }
  g.supported = true;
}

// Per-chiplet element counts of rectangles of one stored operand.
struct Placed {
  int64_t R, Cc;      // logical shape
  bool trans;         // stored as the transpose (Cc x R row-major)
  Placement pl;
  const Layout* lay;
  int G;
  int64_t page;
  int64_t n_pages;    // pages of the stored row-major tensor
  int64_t e;          // element bytes

  int chip_of_page(int64_t pg) const {
    if (pl == PLACE_RR) return (int)(pg % G);
    return (int)((pg * (int64_t)G) / n_pages);   // coarse: G contiguous chunks
  }

  // Bytes [s0, s1) of the stored tensor, split at page boundaries.
  void add_interval(int64_t s0, int64_t s1, uint64_t* h) const {
    int64_t pg = s0 / page;
    while (s0 < s1) {
      int64_t end = std::min((pg + 1) * page, s1);
      h[chip_of_page(pg)] += (uint64_t)((end - s0) / e);
      s0 = end;
      ++pg;
    }
  }

  // Add per-chiplet counts of logical rectangle [r0,r1) x [c0,c1) to h.
  void count(int64_t r0, int64_t r1, int64_t c0, int64_t c1, uint64_t* h) const {
    if (pl == PLACE_CCL) {
      const int64_t hr = lay->block_rows, wc = lay->block_cols;
      for (int64_t br = r0 / hr; br * hr < r1; ++br) {
        int64_t ro = std::min(r1, (br + 1) * hr) - std::max(r0, br * hr);
        for (int64_t bc = c0 / wc; bc * wc < c1; ++bc) {
          int64_t co = std::min(c1, (bc + 1) * wc) - std::max(c0, bc * wc);
          h[br * lay->grid_c + bc] += (uint64_t)(ro * co);
        }
      }
      return;
    }
    if (!trans) {
      for (int64_t r = r0; r < r1; ++r)
        add_interval((r * Cc + c0) * e, (r * Cc + c1) * e, h);
    } else {
      for (int64_t c = c0; c < c1; ++c)
        add_interval((c * R + r0) * e, (c * R + r1) * e, h);
    }
  }
};

}  // namespace

bool grid_aligned(int64_t M, int64_t N, int64_t K, int G, int Gr) {
  if (Gr <= 0 || G % Gr != 0) return false;
  int Gc = G / Gr;
  return M % ((int64_t)Gr * kModelTile) == 0 && N % ((int64_t)Gc * kModelTile) == 0 &&
         K % Gr == 0 && K % Gc == 0;
}

uint64_t floor_bytes(int64_t M, int64_t N, int64_t K, int Gr, int Gc, int ea, int eb) {
  // A: each element read by Gc chiplets, N/(Gc*128) times each, one of them local.
  unsigned __int128 a = (unsigned __int128)M * K * (N / ((int64_t)Gc * kModelTile)) * (Gc - 1) * ea;
  unsigned __int128 b = (unsigned __int128)K * N * (M / ((int64_t)Gr * kModelTile)) * (Gr - 1) * eb;
  return (uint64_t)(a + b);
}

Status make_plan(int64_t M, int64_t N, int64_t K, int chiplets, int grid_rows, int64_t page,
                 DType ab, DType c, Plan* out, std::string* err) {
  if (!out) {
    *err = "plan output pointer is NULL";
    return Status::INVALID_ARG;
  }
  if (M <= 0 || N <= 0 || K <= 0) {
    *err = "M, N and K must be positive";
    return Status::INVALID_ARG;
  }
  const int64_t lim = (int64_t)1 << 31;
  if (M >= lim || N >= lim || K >= lim ||
      (unsigned __int128)M * N * K >= ((unsigned __int128)1 << 62) ||
      (unsigned __int128)M * K >= ((unsigned __int128)1 << 40) ||
      (unsigned __int128)K * N >= ((unsigned __int128)1 << 40) ||
      (unsigned __int128)M * N >= ((unsigned __int128)1 << 40)) {
    *err = "problem size overflows the 64-bit byte counts";
    return Status::INVALID_ARG;
  }
  if (chiplets < 1 || chiplets > kMaxChiplets) {
    *err = "chiplets must be in 1..64";
    return Status::INVALID_ARG;
  }
  if (!is_pow2(page) || page < 128 || page > ((int64_t)1 << 40)) {
    *err = "page_bytes must be a power of two in [128, 2^40]";
    return Status::INVALID_ARG;
  }
  if ((ab != DT_BF16 && ab != DT_FP8_E4M3 && ab != DT_FP32) || (c != DT_BF16 && c != DT_FP32)) {
    *err = "A and B must be bf16, fp8 E4M3 or fp32, C bf16 or fp32";
    return Status::INVALID_ARG;
  }
  const int ea = dtype_bytes(ab), ec = dtype_bytes(c);
  if (grid_rows < 0 || (grid_rows > 0 && chiplets % grid_rows != 0)) {
    *err = "grid_rows must be 0 (automatic) or divide chiplets";
    return Status::INVALID_ARG;
  }
  int Gr = grid_rows;
  if (Gr == 0) {
    // Fewest CCL remote bytes (= floor), then fewest replicated shared
    // bytes, then the smaller grid_rows.
    bool found = false;
    uint64_t best_floor = 0;
    unsigned __int128 best_rep = 0;
    for (int r = 1; r <= chiplets; ++r) {
      if (!grid_aligned(M, N, K, chiplets, r)) continue;
      uint64_t f = floor_bytes(M, N, K, r, chiplets / r, ea, ea);
      unsigned __int128 rep = replicated_times_g(M, N, K, r, chiplets / r, ea, ea);
      if (!found || f < best_floor || (f == best_floor && rep < best_rep)) {
        found = true;
        best_floor = f;
        best_rep = rep;
        Gr = r;
      }
    }
    if (!found) {
      *err = "no grid gives 128-aligned partitions";
      return Status::UNALIGNED;
    }
  } else if (!grid_aligned(M, N, K, chiplets, Gr)) {
    *err = "partitions must be multiples of 128x128 tiles and K divisible by both grid sides";
    return Status::UNALIGNED;
  }
  Plan p;
  p.M = M;
  p.N = N;
  p.K = K;
  p.G = chiplets;
  p.Gr = Gr;
  p.Gc = chiplets / Gr;
  p.page = page;
  p.ab_type = ab;
  p.c_type = c;
  p.lay[OP_A] = make_layout(M, K, p.Gr, p.Gc, page, ea);
  p.lay[OP_B] = make_layout(K, N, p.Gr, p.Gc, page, ea);
  p.lay[OP_C] = make_layout(M, N, p.Gr, p.Gc, page, ec);
  choose_gemm_config(&p);
  *out = p;
  return Status::OK;
}

Traffic remote_bytes(const Plan& p, Placement pl, int flags) {
  const int trans_mask = flags & 3;
  const uint64_t c_times = (flags & kTrafficCRead) ? 2 : 1;   // beta != 0: C read, then written
  Traffic t;
  t.chiplets = p.G;
  const int G = p.G;
  const int64_t T = kModelTile;
  const int64_t TM = p.M / T, TN = p.N / T;
  const int64_t tm_per_part = p.part_rows() / T, tn_per_part = p.part_cols() / T;
  const int64_t shapes[3][2] = {{p.M, p.K}, {p.K, p.N}, {p.M, p.N}};
  Placed ops[3];
  for (int o = 0; o < 3; ++o) {
    const int64_t e = p.lay[o].elem_bytes;
    int64_t bytes = shapes[o][0] * shapes[o][1] * e;
    ops[o] = Placed{shapes[o][0], shapes[o][1], o < 2 && ((trans_mask >> o) & 1), pl,
                    &p.lay[o],   G,            p.page, (bytes + p.page - 1) / p.page, e};
    t.footprint[o] = pl == PLACE_CCL ? (uint64_t)p.lay[o].total_bytes : (uint64_t)bytes;
  }
  std::vector<uint64_t> h(G);
  const uint64_t ea = p.lay[OP_A].elem_bytes, eb = p.lay[OP_B].elem_bytes, ec = p.lay[OP_C].elem_bytes;

  // A: row panel ti is read by the TN tiles of its row; the tiles of grid
  // column pc are owned by chiplet pr*Gc + pc, tn_per_part of them.
  for (int64_t ti = 0; ti < TM; ++ti) {
    std::fill(h.begin(), h.end(), 0);
    ops[OP_A].count(ti * T, (ti + 1) * T, 0, p.K, h.data());
    const int pr = (int)(ti / tm_per_part);
    for (int pc = 0; pc < p.Gc; ++pc) {
      const int o = pr * p.Gc + pc;
      uint64_t rem = ea * (uint64_t)tn_per_part * ((uint64_t)(T * p.K) - h[o]);
      t.remote[OP_A] += rem;
      t.remote_per_chiplet[o] += rem;
    }
  }
  // B: column panel tj is read by the TM tiles of its column.
  for (int64_t tj = 0; tj < TN; ++tj) {
    std::fill(h.begin(), h.end(), 0);
    ops[OP_B].count(0, p.K, tj * T, (tj + 1) * T, h.data());
    const int pc = (int)(tj / tn_per_part);
    for (int pr = 0; pr < p.Gr; ++pr) {
      const int o = pr * p.Gc + pc;
      uint64_t rem = eb * (uint64_t)tm_per_part * ((uint64_t)(p.K * T) - h[o]);
      t.remote[OP_B] += rem;
      t.remote_per_chiplet[o] += rem;
    }
  }
  // C: each tile written once by its owner (and read once before that when
  // c_times == 2; the read has the write's partitioning).
  for (int64_t ti = 0; ti < TM; ++ti) {
    for (int64_t tj = 0; tj < TN; ++tj) {
      std::fill(h.begin(), h.end(), 0);
      ops[OP_C].count(ti * T, (ti + 1) * T, tj * T, (tj + 1) * T, h.data());
      const int o = p.owner(ti, tj);
      uint64_t rem = c_times * ec * ((uint64_t)(T * T) - h[o]);
      t.remote[OP_C] += rem;
      t.remote_per_chiplet[o] += rem;
    }
  }
  t.accessed[OP_A] = ea * (uint64_t)p.M * p.K * TN;
  t.accessed[OP_B] = eb * (uint64_t)p.K * p.N * TM;
  t.accessed[OP_C] = c_times * ec * (uint64_t)p.M * p.N;
  t.floor_bytes = floor_bytes(p.M, p.N, p.K, p.Gr, p.Gc, (int)ea, (int)eb);
  return t;
}

TileMap tile_map(const Plan& p, int splits) {
  const GemmConfig& g = p.gemm;
  const int64_t per_xcd = (g.tiles_m * g.tiles_n * splits + g.xcd_per_chiplet - 1) / g.xcd_per_chiplet;
  return TileMap{g.xcd_per_chiplet, p.Gc, (int32_t)g.tiles_m, (int32_t)g.tiles_n,
                 (int32_t)per_xcd, g.group_m, splits};
}

int64_t gemm_ksteps(const Plan& p) {
  return p.K / (p.ab_type == DT_FP8_E4M3 ? kGemmBK8 : kGemmBK);
}

int recommended_splits(const Plan& p) {
  const GemmConfig& g = p.gemm;
  if (!g.supported) return 1;
  // Fill the XCD's 32 CUs when its partition has few tiles, keeping at
  // least 8 K steps per split.
  const int64_t per_xcd = g.tiles_per_xcd;
  int s = (int)std::max<int64_t>(1, 32 / std::max<int64_t>(1, per_xcd));
  s = (int)std::min<int64_t>(s, std::max<int64_t>(1, gemm_ksteps(p) / 8));
  return std::min(s, kMaxSplits);
}

int effective_splits(const Plan& p, int splits) {
  const int64_t ks = gemm_ksteps(p);
  if (splits <= 1 || ks <= 1) return 1;
  const int64_t per = (ks + splits - 1) / splits;
  return (int)((ks + per - 1) / per);
}

int64_t splitk_workgroups(const Plan& p, int splits) {
  const GemmConfig& g = p.gemm;
  const int64_t tiles = g.tiles_m * g.tiles_n * effective_splits(p, splits);
  return kNumXcd * ((tiles + g.xcd_per_chiplet - 1) / g.xcd_per_chiplet);
}

int64_t splitk_reduce_workgroups(const Plan& p) {
  const GemmConfig& g = p.gemm;
  return g.workgroups * (g.tile_m * g.tile_n / 1024);
}

int64_t splitk_workspace_bytes(const Plan& p, int splits) {
  const GemmConfig& g = p.gemm;
  const int s = effective_splits(p, splits);
  return s > 1 ? (int64_t)p.G * g.tiles_m * g.tiles_n * s * g.tile_m * g.tile_n * 4 : 0;
}

void tile_of_wg(const Plan& p, int64_t wg, int* xcd, int64_t* tile_m, int64_t* tile_n) {
  *xcd = (int)(wg % kNumXcd);
  *tile_m = *tile_n = -1;
  if (!p.gemm.supported || wg < 0 || wg >= p.gemm.workgroups) return;
  int32_t pr, pc, ti, tj;
  if (!map_tile(tile_map(p), wg, &pr, &pc, &ti, &tj)) return;
  *tile_m = (int64_t)pr * p.gemm.tiles_m + ti;
  *tile_n = (int64_t)pc * p.gemm.tiles_n + tj;
}

}  // namespace ccl
