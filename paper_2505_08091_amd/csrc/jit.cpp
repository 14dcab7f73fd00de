// hipRTC compilation and code-object caching.  See jit.hpp.
#include "jit.hpp"

#include <dlfcn.h>
#include <hip/hiprtc.h>
#include <sys/stat.h>
#include <unistd.h>

#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <fstream>
#include <map>
#include <mutex>
#include <sstream>
#include <stdexcept>

namespace lego {

namespace {

std::mutex g_mu;
std::map<std::string, JitKernel> g_mem;         // key + device + name -> function
std::map<std::string, hipModule_t> g_modules;   // key + device -> module
JitStats g_stats;

// hipRTC of the installed ROCm (ROCM_PATH, default /opt/rocm), loaded into a
// link namespace of its own.  hipRTC opens its compiler library (comgr) by
// soname at run time; a host process that already carries another ROCm
// release's comgr (a PyTorch wheel bundles one) would otherwise hand it that
// older compiler, whose code for the one-wave-per-SIMD GEMM spills its
// accumulators to scratch.  The namespace keeps the installed compiler.  If
// the private load fails, the hipRTC the process resolves normally is used.
struct Rtc {
  hiprtcResult (*version)(int*, int*);
  hiprtcResult (*create)(hiprtcProgram*, const char*, const char*, int, const char**, const char**);
  hiprtcResult (*compile)(hiprtcProgram, int, const char**);
  hiprtcResult (*log_size)(hiprtcProgram, size_t*);
  hiprtcResult (*log)(hiprtcProgram, char*);
  hiprtcResult (*code_size)(hiprtcProgram, size_t*);
  hiprtcResult (*code)(hiprtcProgram, char*);
  hiprtcResult (*destroy)(hiprtcProgram*);
  std::string origin;
};

const Rtc& rtc() {
  static const Rtc r = [] {
    const char* root = std::getenv("ROCM_PATH");
    std::string path = std::string(root && *root ? root : "/opt/rocm") + "/lib/libhiprtc.so.7";
    void* h = dlmopen(LM_ID_NEWLM, path.c_str(), RTLD_NOW | RTLD_LOCAL);
    std::string origin = path + " (private namespace)";
    if (!h) {
      h = dlopen("libhiprtc.so.7", RTLD_NOW | RTLD_LOCAL);
      origin = "libhiprtc.so.7 (process namespace)";
    }
    if (!h) throw std::runtime_error("hipRTC library not found");
    auto sym = [&](const char* name) {
      void* f = dlsym(h, name);
      if (!f) throw std::runtime_error(std::string("hipRTC symbol missing: ") + name);
      return f;
    };
    Rtc t;
    t.version = (decltype(t.version))sym("hiprtcVersion");
    t.create = (decltype(t.create))sym("hiprtcCreateProgram");
    t.compile = (decltype(t.compile))sym("hiprtcCompileProgram");
    t.log_size = (decltype(t.log_size))sym("hiprtcGetProgramLogSize");
    t.log = (decltype(t.log))sym("hiprtcGetProgramLog");
    t.code_size = (decltype(t.code_size))sym("hiprtcGetCodeSize");
    t.code = (decltype(t.code))sym("hiprtcGetCode");
    t.destroy = (decltype(t.destroy))sym("hiprtcDestroyProgram");
    t.origin = origin;
    return t;
  }();
  return r;
}

}  // namespace

std::string jit_compiler() {
  int major = 0, minor = 0;
  rtc().version(&major, &minor);
  return "hipRTC " + std::to_string(major) + "." + std::to_string(minor) + " from " + rtc().origin;
}

namespace {

uint64_t fnv1a(const std::string& s, uint64_t h = 1469598103934665603ull) {
  for (unsigned char ch : s) {
    h ^= ch;
    h *= 1099511628211ull;
  }
  return h;
}

std::string hex(uint64_t v) {
  char b[17];
  std::snprintf(b, sizeof b, "%016llx", (unsigned long long)v);
  return b;
}

std::string cache_dir() {
  const char* d = std::getenv("LEGO_CACHE_DIR");
  if (d && *d) return d;
  const char* home = std::getenv("HOME");
  if (!home || !*home) return "";
  return std::string(home) + "/.cache/lego_mi355x";
}

void mkdirs(const std::string& path) {
  std::string cur;
  std::stringstream ss(path);
  std::string part;
  if (!path.empty() && path[0] == '/') cur = "/";
  while (std::getline(ss, part, '/')) {
    if (part.empty()) continue;
    cur += part + "/";
    mkdir(cur.c_str(), 0755);
  }
}

std::string source_key(const std::string& src) {
  int major = 0, minor = 0;
  rtc().version(&major, &minor);
  std::string k = src;
  for (auto& o : jit_options()) k += "\x1f" + o;
  k += "\x1fhiprtc" + std::to_string(major) + "." + std::to_string(minor);
  return hex(fnv1a(k)) + hex(fnv1a(k, 0x9e3779b97f4a7c15ull));
}

bool read_file(const std::string& p, std::vector<char>* out) {
  std::ifstream f(p, std::ios::binary);
  if (!f) return false;
  out->assign(std::istreambuf_iterator<char>(f), std::istreambuf_iterator<char>());
  return !out->empty();
}

void write_file_atomic(const std::string& p, const std::vector<char>& data) {
  std::string tmp = p + ".tmp" + std::to_string(getpid());
  {
    std::ofstream f(tmp, std::ios::binary);
    if (!f) return;
    f.write(data.data(), (std::streamsize)data.size());
    if (!f) return;
  }
  std::rename(tmp.c_str(), p.c_str());
}

// A cached code object carries a trailing 16-hex-digit checksum of its bytes,
// so a truncated or corrupted entry is detected and recompiled.
bool unpack_cached(std::vector<char>* blob) {
  if (blob->size() < 17) return false;
  std::string tail(blob->end() - 16, blob->end());
  blob->resize(blob->size() - 16);
  return hex(fnv1a(std::string(blob->begin(), blob->end()))) == tail;
}

void pack_cached(std::vector<char>* blob) {
  std::string h = hex(fnv1a(std::string(blob->begin(), blob->end())));
  blob->insert(blob->end(), h.begin(), h.end());
}

}  // namespace

const std::vector<std::string>& jit_options() {
  static const std::vector<std::string> opts = [] {
    std::vector<std::string> o = {
        "--offload-arch=gfx950", "-O3", "-std=c++17",
        // Packed fp32 instructions are disabled for all generated code.
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    };
    // Extra compiler options for tuning experiments (space separated).
    if (const char* extra = std::getenv("LEGO_JIT_OPTS")) {
      std::istringstream ss(extra);
      std::string w;
      while (ss >> w) o.push_back(w);
    }
    return o;
  }();
  return opts;
}

std::vector<char> jit_compile(const std::string& src, std::string* log, double* ms) {
  auto t0 = std::chrono::steady_clock::now();
  if (const char* dump = std::getenv("LEGO_DUMP")) {
    // Keep every generated source for inspection.
    if (*dump) {
      mkdirs(dump);
      std::ofstream f(std::string(dump) + "/" + source_key(src) + ".hip");
      f << src;
    }
  }
  const Rtc& R = rtc();
  hiprtcProgram prog;
  if (R.create(&prog, src.c_str(), "lego_generated.hip", 0, nullptr, nullptr) != HIPRTC_SUCCESS)
    throw std::runtime_error("hiprtcCreateProgram failed");
  std::vector<const char*> o;
  for (auto& s : jit_options()) o.push_back(s.c_str());
  hiprtcResult rc = R.compile(prog, (int)o.size(), o.data());
  size_t n = 0;
  R.log_size(prog, &n);
  std::string lg(n, '\0');
  if (n) R.log(prog, &lg[0]);
  if (log) *log = lg;
  if (rc != HIPRTC_SUCCESS) {
    R.destroy(&prog);
    throw std::runtime_error("hipRTC compilation failed:\n" + lg);
  }
  size_t cs = 0;
  R.code_size(prog, &cs);
  std::vector<char> code(cs);
  R.code(prog, code.data());
  R.destroy(&prog);
  if (const char* dump = std::getenv("LEGO_DUMP")) {
    if (*dump) {
      mkdirs(dump);
      std::ofstream f(std::string(dump) + "/" + source_key(src) + ".co", std::ios::binary);
      f.write(code.data(), (std::streamsize)code.size());
    }
  }
  auto t1 = std::chrono::steady_clock::now();
  if (ms) *ms = std::chrono::duration<double, std::milli>(t1 - t0).count();
  return code;
}

JitKernel jit_get(const std::string& src, const std::string& name) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) throw std::runtime_error("no HIP device");
  std::string key = source_key(src);
  std::string mkey = key + "@" + std::to_string(dev);
  std::lock_guard<std::mutex> lk(g_mu);
  auto hit = g_mem.find(mkey + ":" + name);
  if (hit != g_mem.end()) {
    ++g_stats.mem_hits;
    JitKernel k = hit->second;
    k.compile_ms = 0;
    return k;
  }
  hipModule_t mod = nullptr;
  double ms = 0;
  auto mit = g_modules.find(mkey);
  if (mit != g_modules.end()) {
    mod = mit->second;
  } else {
    std::vector<char> code;
    std::string dir = cache_dir();
    std::string path = dir.empty() ? "" : dir + "/" + key + ".co";
    bool have = false;
    if (!path.empty() && read_file(path, &code) && unpack_cached(&code)) {
      have = hipModuleLoadData(&mod, code.data()) == hipSuccess;
      if (have) ++g_stats.disk_hits;
    }
    if (!have) {
      std::string log;
      code = jit_compile(src, &log, &ms);
      ++g_stats.compiles;
      g_stats.compile_ms += ms;
      hipError_t e = hipModuleLoadData(&mod, code.data());
      if (e != hipSuccess) throw std::runtime_error(std::string("hipModuleLoadData: ") + hipGetErrorString(e));
      if (!path.empty()) {
        mkdirs(dir);
        std::vector<char> blob = code;
        pack_cached(&blob);
        write_file_atomic(path, blob);
      }
    }
    g_modules[mkey] = mod;
  }
  JitKernel k;
  hipError_t e = hipModuleGetFunction(&k.fn, mod, name.c_str());
  if (e != hipSuccess) throw std::runtime_error("kernel " + name + " not found in generated module");
  k.compile_ms = ms;
  JitKernel stored = k;
  g_mem[mkey + ":" + name] = stored;
  return k;
}

JitStats jit_stats() {
  std::lock_guard<std::mutex> lk(g_mu);
  return g_stats;
}

}  // namespace lego
