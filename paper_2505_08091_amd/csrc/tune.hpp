// Planner experiment switch.  LEGO_TUNE="key=value,key=value" overrides the
// measured defaults of individual planner choices (for timing experiments
// only; it is read once per process, is not part of the C ABI, and every
// default is what the measurements chose).  Keys: gemm.lds_s, gemm.mfma,
// gemm.direct, gemm.prefetch, gemm.rolling, gemm.dma_spread, gemm.frag_dist,
// gemm.frag_spread, gemm.store_at, gemm.persist, gemm.ring_unroll, gemm.wide_waves, gemm.zdirect, gemm.zpair,
// gemm.dma_rows, index.nt_store, index.grid, remap.nontemporal, remap.box,
// remap.box_side, remap.box_tile, remap.box_band, remap.nt, remap.unroll, remap.order (0 destination, 1
// source), remap.xcd, remap.persist, remap.tile_bytes, remap.block (LDS block
// transfer), remap.swizzle, remap.swizzle2, remap.lds_row (LDS XOR key strides
// and row bytes).
#pragma once

#include <cstdlib>
#include <map>
#include <string>

namespace lego {

inline const std::map<std::string, long long>& tune_table() {
  static const std::map<std::string, long long> table = [] {
    std::map<std::string, long long> t;
    const char* e = std::getenv("LEGO_TUNE");
    if (!e) return t;
    std::string s(e);
    size_t i = 0;
    while (i < s.size()) {
      size_t j = s.find(',', i);
      if (j == std::string::npos) j = s.size();
      const std::string kv = s.substr(i, j - i);
      const size_t eq = kv.find('=');
      if (eq != std::string::npos) t[kv.substr(0, eq)] = std::atoll(kv.c_str() + eq + 1);
      i = j + 1;
    }
    return t;
  }();
  return table;
}

// The value set for `key`, or `def`.
inline long long tune(const char* key, long long def) {
  const auto& t = tune_table();
  auto it = t.find(key);
  return it == t.end() ? def : it->second;
}

}  // namespace lego
