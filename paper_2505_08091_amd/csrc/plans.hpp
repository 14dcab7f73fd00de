// Kernel planning: from layouts to a generated source, a kernel name and a
// launch shape.  Planning needs no GPU (the build check compiles every plan's
// source for gfx950); launching does.
#pragma once

#include <mutex>
#include <string>
#include <vector>

#include "layout.hpp"

namespace lego {

// Loaded kernel functions of one plan object, per device ordinal, so that a
// launch of a cached plan skips hashing its source.  A copy starts empty: the
// copy may be edited into a different source.
struct FnCache {
  static constexpr int kDevices = 64;
  FnCache() = default;
  FnCache(const FnCache&) {}
  FnCache& operator=(const FnCache&) {
    std::lock_guard<std::mutex> lk(mu);
    for (auto& f : fn) f = nullptr;
    for (auto& r : resident) r = 0;
    return *this;
  }
  mutable std::mutex mu;
  mutable void* fn[kDevices] = {};
  mutable long long resident[kDevices] = {};  // workgroups resident at once (persistent plans)
};

struct KernelPlan {
  std::string src;      // complete generated HIP source
  std::string kernel;   // extern "C" kernel name
  long long grid = 1;   // workgroups (1D)
  int block = 256;      // threads per workgroup
  std::string info;     // human-readable summary (path, vector widths, op counts)
  bool persistent = false;  // the kernel walks tiles grid-stride: launch at most
                            // as many workgroups as fit on the device at once
  FnCache fns;          // filled by the first launch on each device
};

// Index-map evaluation over all points: which = 0 apply (logical flat order),
// which = 1 inv (physical order, `rank` outputs per point).
KernelPlan plan_index_eval(const Layout& l, int which, int idx_bytes);

enum RemapPath { REMAP_DIRECT = 0, REMAP_LDS = 1, REMAP_GATHER = 2, REMAP_BOX = 3 };

struct RemapPlan : KernelPlan {
  int path = REMAP_GATHER;
  long long run = 1;    // contiguous run of M (elements)
  int vec = 1;          // elements per vector (direct) or source-side vector (LDS)
  int vec_dst = 1;      // destination-side vector (LDS)
  long long tile = 0;   // elements per LDS tile
};

RemapPlan plan_remap(const Layout& src, const Layout& dst, int elem_bytes);

// Template texts, embedded at build time from csrc/kernels/*.hip.
extern const char* const tpl_index_eval;
extern const char* const tpl_remap;
extern const char* const tpl_gemm;

}  // namespace lego
