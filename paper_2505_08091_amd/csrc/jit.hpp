// Runtime compilation of generated kernel sources for gfx950 with hipRTC.
//
// A generated source (the prelude, the emitted index functions and a kernel
// template) is compiled once per process and device; code objects are also
// kept on disk under $LEGO_CACHE_DIR (default ~/.cache/lego_mi355x), keyed by
// a hash of the source text, the compile options and the hipRTC version, so a
// later process loads instead of compiling.  Compilation is excluded from the
// steady state, as the paper excludes code generation (Table III).
#pragma once

#include <hip/hip_runtime.h>

#include <string>
#include <vector>

namespace lego {

struct JitKernel {
  hipFunction_t fn = nullptr;
  double compile_ms = 0;  // 0 when served from a cache
};

// Compile (or fetch) `src` and return kernel `name` loaded on the current
// device.  Throws std::runtime_error with the compiler log on failure.
JitKernel jit_get(const std::string& src, const std::string& name);

// Compile only (no device needed); returns the code object.  Used by the
// build check to prove every generated source compiles for gfx950.
std::vector<char> jit_compile(const std::string& src, std::string* log, double* ms);

// Options passed to hipRTC (also recorded in the cache key).
const std::vector<std::string>& jit_options();

// "hipRTC <major>.<minor> from <library> (<namespace>)": the compiler behind
// jit_compile.
std::string jit_compiler();

struct JitStats {
  long compiles = 0, disk_hits = 0, mem_hits = 0;
  double compile_ms = 0;
};
JitStats jit_stats();

}  // namespace lego
