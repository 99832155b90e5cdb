// Remote-HBM traffic of a CCL plan's GEMM with a private set-associative LRU
// L2 per chiplet (Sec. IV-A simulation framework). Plain C++17, host only.
#pragma once

#include <cstdint>
#include <string>

#include "plan.hpp"

namespace ccl {

struct L2Config {
  int64_t l2_bytes = 0;   // per chiplet; 0 = no cache (every access misses)
  int ways = 16;
  int line = 128;         // bytes, power of two
  int slots = 32;         // tiles resident per chiplet at once
  int k_step = 64;        // K elements each resident tile reads per step
  int traversal = 0;      // 0: tile rows outer, 1: tile columns outer, 2: grouped raster
  int group_rows = 0;     // traversal 2: tile rows per group (each group walked column by column)
  int threads = 0;        // host threads (0: one per chiplet, up to the core count)
};

struct L2Traffic {
  uint64_t accesses[2] = {0, 0};   // A, B line accesses
  uint64_t misses[2] = {0, 0};
  uint64_t remote[3] = {0, 0, 0};  // bytes: A, B remote misses; C remote line writes
  uint64_t remote_per_chiplet[kMaxChiplets] = {};
  int chiplets = 0;
};

// Validate a configuration; empty string when usable.
std::string check_l2_config(const L2Config& c);

// flags as for remote_bytes (plan.hpp).
L2Traffic remote_bytes_l2(const Plan& p, Placement pl, int flags, const L2Config& c);

}  // namespace ccl
