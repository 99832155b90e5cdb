// Finite-L2 remote-traffic model (Sec. IV-A simulation framework).
//
// Each chiplet runs the 128x128 tiles of its own partition, `slots` at a
// time, in the chosen traversal order. The tiles of one wave step through K
// together, k_step elements at a time; at each step every tile of the wave,
// in wave order, reads the lines of its A slice and then of its B slice, in
// increasing address order of the operand as stored. Each line access goes
// through the chiplet's private L2: `sets` sets of `ways` lines, the set
// being the line number folded by XOR into log2(sets) bits, true LRU within
// a set. A miss is remote when the line's home chiplet under the placement is
// not the one running the tile. When a wave has finished K, each of its tiles
// writes its C tile, which is not cached; each C line homed elsewhere costs
// one line of remote traffic (two when C is also read, beta != 0).
//
// Chiplets have private caches and are simulated independently, one host
// thread each.
#include "l2sim.hpp"

#include <algorithm>
#include <atomic>
#include <cstring>
#include <thread>
#include <vector>

namespace ccl {

namespace {

enum Storage { ROW_MAJOR = 0, TRANSPOSED = 1, CCL_STRIPS = 2 };

// How one operand is stored and where its pages live.
struct Stored {
  Storage kind = ROW_MAJOR;
  int64_t R = 0, C = 0;              // logical rows, cols
  int64_t hr = 1, wc = 1, S = 0;     // CCL block rows / cols, strip stride (bytes)
  int Pc = 1;
  Placement place = PLACE_RR;
  int G = 1;
  int64_t page = 4096, n_pages = 1;
  int64_t e = 2;                     // element bytes
  uint64_t base_line = 0;            // line number of the buffer's first byte

  int home(int64_t off) const {
    if (place == PLACE_CCL) return static_cast<int>(off / S);
    const int64_t pg = off / page;
    if (place == PLACE_RR) return static_cast<int>(pg % G);
    return static_cast<int>(pg * G / n_pages);
  }
};

Stored make_stored(const Plan& p, Op op, Placement pl, bool trans, int line) {
  const Layout& L = p.lay[op];
  Stored s;
  s.R = L.rows;
  s.C = L.cols;
  s.place = pl;
  s.G = p.G;
  s.page = p.page;
  s.e = L.elem_bytes;
  if (pl == PLACE_CCL) {
    s.kind = CCL_STRIPS;
    s.hr = L.block_rows;
    s.wc = L.block_cols;
    s.Pc = static_cast<int>(L.grid_c);
    s.S = L.strip_stride_bytes;
  } else {
    s.kind = trans ? TRANSPOSED : ROW_MAJOR;
    s.n_pages = (L.rows * L.cols * L.elem_bytes + p.page - 1) / p.page;
  }
  s.base_line = (uint64_t(op) << 40) / uint64_t(line);   // A at 0, B at 2^40, C at 2^41
  return s;
}

// Calls f(byte offset of the line's first byte) for every distinct line the
// logical slice rows [r0, r1) x cols [c0, c1) touches, in increasing order.
// The byte runs below are produced in increasing address order, so a line
// shared by consecutive runs is the last one emitted.
template <typename F>
void for_each_line(const Stored& s, int64_t r0, int64_t r1, int64_t c0, int64_t c1, int line_shift,
                   F&& f) {
  int64_t last = -1;
  auto run = [&](int64_t begin, int64_t end) {       // bytes [begin, end)
    int64_t l = begin >> line_shift;
    if (l == last) ++l;
    const int64_t l1 = (end - 1) >> line_shift;
    for (; l <= l1; ++l) f(l << line_shift);
    last = l1;
  };
  const int64_t e = s.e;
  switch (s.kind) {
    case ROW_MAJOR:
      for (int64_t r = r0; r < r1; ++r) run((r * s.C + c0) * e, (r * s.C + c1) * e);
      break;
    case TRANSPOSED:                                 // stored C x R
      for (int64_t c = c0; c < c1; ++c) run((c * s.R + r0) * e, (c * s.R + r1) * e);
      break;
    case CCL_STRIPS:
      for (int64_t br = r0 / s.hr; br <= (r1 - 1) / s.hr; ++br) {
        for (int64_t bc = c0 / s.wc; bc <= (c1 - 1) / s.wc; ++bc) {
          const int64_t strip = (br * s.Pc + bc) * s.S;
          const int64_t lr0 = std::max(r0, br * s.hr) - br * s.hr;
          const int64_t lr1 = std::min(r1, (br + 1) * s.hr) - br * s.hr;
          const int64_t lc0 = std::max(c0, bc * s.wc) - bc * s.wc;
          const int64_t lc1 = std::min(c1, (bc + 1) * s.wc) - bc * s.wc;
          for (int64_t lr = lr0; lr < lr1; ++lr)
            run(strip + (lr * s.wc + lc0) * e, strip + (lr * s.wc + lc1) * e);
        }
      }
      break;
  }
}

// Set-associative LRU cache of line numbers; each set's lines are kept most
// recent first.
class Lru {
 public:
  Lru(int64_t capacity_bytes, int ways, int line) : ways_(ways) {
    if (capacity_bytes == 0) return;
    on_ = true;
    const int64_t sets = capacity_bytes / (int64_t(line) * ways);
    while ((int64_t(1) << bits_) < sets) ++bits_;
    mask_ = (uint64_t(1) << bits_) - 1;
    tags_.assign(size_t(sets) * ways, 0);
    count_.assign(size_t(sets), 0);
  }

  bool access(uint64_t line) {
    if (!on_) return false;
    const uint64_t set = fold(line);
    uint64_t* t = tags_.data() + set * ways_;
    int& n = count_[set];
    for (int i = 0; i < n; ++i) {
      if (t[i] == line) {
        std::memmove(t + 1, t, sizeof(uint64_t) * i);
        t[0] = line;
        return true;
      }
    }
    const int keep = n < ways_ ? n : ways_ - 1;
    std::memmove(t + 1, t, sizeof(uint64_t) * keep);
    t[0] = line;
    if (n < ways_) ++n;
    return false;
  }

 private:
  uint64_t fold(uint64_t line) const {
    if (bits_ == 0) return 0;
    uint64_t x = 0;
    for (; line; line >>= bits_) x ^= line & mask_;
    return x;
  }

  bool on_ = false;
  int ways_;
  int bits_ = 0;
  uint64_t mask_ = 0;
  std::vector<uint64_t> tags_;
  std::vector<int> count_;
};

struct ChipletCount {
  uint64_t accesses[2] = {0, 0}, misses[2] = {0, 0}, remote[3] = {0, 0, 0};
};

ChipletCount simulate_chiplet(const Plan& p, int chip, const Stored* st, const L2Config& c,
                              uint64_t c_times) {
  ChipletCount out;
  Lru cache(c.l2_bytes, c.ways, c.line);
  int shift = 0;
  while ((1 << shift) < c.line) ++shift;
  const int64_t TR = p.M / (p.Gr * int64_t(kModelTile)), TC = p.N / (p.Gc * int64_t(kModelTile));
  const int64_t pr = chip / p.Gc, pc = chip % p.Gc;
  const int64_t ntiles = TR * TC;
  const int64_t nk = (p.K + c.k_step - 1) / c.k_step;
  auto tile = [&](int64_t t, int64_t* ti, int64_t* tj) {
    if (c.traversal == 0) {
      *ti = pr * TR + t / TC;
      *tj = pc * TC + t % TC;
    } else if (c.traversal == 1) {
      *tj = pc * TC + t / TR;
      *ti = pr * TR + t % TR;
    } else {
      // groups of group_rows tile rows (the last one may be shorter), each
      // walked column by column down its rows
      const int64_t per_group = int64_t(c.group_rows) * TC;
      const int64_t first = (t / per_group) * c.group_rows;
      const int64_t gm = std::min<int64_t>(c.group_rows, TR - first);
      const int64_t w = t - (t / per_group) * per_group;
      *ti = pr * TR + first + w % gm;
      *tj = pc * TC + w / gm;
    }
  };
  const int64_t T = kModelTile;
  for (int64_t w0 = 0; w0 < ntiles; w0 += c.slots) {
    const int64_t wn = std::min<int64_t>(c.slots, ntiles - w0);
    for (int64_t s = 0; s < nk; ++s) {
      const int64_t k0 = s * c.k_step, k1 = std::min<int64_t>(p.K, k0 + c.k_step);
      for (int64_t j = 0; j < wn; ++j) {
        int64_t ti, tj;
        tile(w0 + j, &ti, &tj);
        for (int op = 0; op < 2; ++op) {
          const Stored& o = st[op];
          auto touch = [&](int64_t off) {
            ++out.accesses[op];
            if (!cache.access(o.base_line + uint64_t(off >> shift))) {
              ++out.misses[op];
              if (o.home(off) != chip) out.remote[op] += uint64_t(c.line);
            }
          };
          if (op == 0)
            for_each_line(o, ti * T, ti * T + T, k0, k1, shift, touch);
          else
            for_each_line(o, k0, k1, tj * T, tj * T + T, shift, touch);
        }
      }
    }
    for (int64_t j = 0; j < wn; ++j) {
      int64_t ti, tj;
      tile(w0 + j, &ti, &tj);
      for_each_line(st[OP_C], ti * T, ti * T + T, tj * T, tj * T + T, shift, [&](int64_t off) {
        if (st[OP_C].home(off) != chip) out.remote[2] += c_times * uint64_t(c.line);
      });
    }
  }
  return out;
}

bool pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

}  // namespace

std::string check_l2_config(const L2Config& c) {
  if (c.line < 16 || !pow2(c.line)) return "line must be a power of two >= 16";
  if (c.ways < 1) return "ways must be >= 1";
  if (c.slots < 1) return "slots must be >= 1";
  if (c.k_step < 1) return "k_step must be >= 1";
  if (c.traversal < 0 || c.traversal > 2)
    return "traversal must be 0 (rows), 1 (columns) or 2 (grouped raster)";
  if (c.traversal == 2 && c.group_rows < 1) return "group_rows must be >= 1 for traversal 2";
  if (c.threads < 0) return "threads must be >= 0";
  if (c.l2_bytes < 0) return "l2_bytes must be >= 0";
  if (c.l2_bytes > 0) {
    const int64_t set_bytes = int64_t(c.line) * c.ways;
    if (c.l2_bytes % set_bytes) return "l2_bytes must be a whole number of sets (line * ways)";
    if (!pow2(c.l2_bytes / set_bytes)) return "the number of sets must be a power of two";
    if (c.l2_bytes / c.line > (int64_t(1) << 24)) return "l2_bytes / line must be <= 2^24";
  }
  return "";
}

L2Traffic remote_bytes_l2(const Plan& p, Placement pl, int flags, const L2Config& c) {
  const int trans_mask = flags & 3;
  const uint64_t c_times = (flags & kTrafficCRead) ? 2 : 1;
  Stored st[3] = {make_stored(p, OP_A, pl, trans_mask & 1, c.line),
                  make_stored(p, OP_B, pl, (trans_mask >> 1) & 1, c.line),
                  make_stored(p, OP_C, pl, false, c.line)};
  std::vector<ChipletCount> per(p.G);
  // Each thread holds one chiplet's tag array (l2_bytes / line * 8 bytes), so
  // never run more threads than there are cores.
  const int cores = static_cast<int>(std::max(1u, std::thread::hardware_concurrency()));
  int nthreads = c.threads == 0 ? cores : std::min(c.threads, cores);
  nthreads = std::min(nthreads, p.G);
  std::atomic<int> next{0};
  auto worker = [&] {
    for (int chip; (chip = next.fetch_add(1)) < p.G;) per[chip] = simulate_chiplet(p, chip, st, c, c_times);
  };
  if (nthreads <= 1) {
    worker();
  } else {
    std::vector<std::thread> pool;
    for (int i = 0; i < nthreads; ++i) pool.emplace_back(worker);
    for (auto& t : pool) t.join();
  }
  L2Traffic t;
  t.chiplets = p.G;
  for (int chip = 0; chip < p.G; ++chip) {
    for (int i = 0; i < 2; ++i) {
      t.accesses[i] += per[chip].accesses[i];
      t.misses[i] += per[chip].misses[i];
    }
    for (int i = 0; i < 3; ++i) {
      t.remote[i] += per[chip].remote[i];
      t.remote_per_chiplet[chip] += per[chip].remote[i];
    }
  }
  return t;
}

}  // namespace ccl
