// The C ABI (include/lego.h): handles, status codes, plan caches, launches.
#include "lego.h"

#include <hip/hip_runtime.h>

#include <atomic>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <sstream>
#include <string>
#include <tuple>
#include <vector>

#include "errors.hpp"
#include "gemm_plan.hpp"
#include "jit.hpp"
#include "lower.hpp"
#include "plans.hpp"

using namespace lego;

struct lego_piece_s {
  uint32_t magic = 0x50434549u;
  std::atomic<int> rc{1};
  PieceP p;
};
struct lego_layout_s {
  uint32_t magic = 0x4c41594fu;
  std::atomic<int> rc{1};
  LayoutP l;
};

namespace {

thread_local std::string g_err;

lego_status fail(lego_status code, const std::string& msg) {
  g_err = msg;
  return code;
}

template <class F>
lego_status guard(F&& f) {
  try {
    g_err.clear();
    return f();
  } catch (const Unsupported& e) {
    return fail(LEGO_E_UNSUPPORTED, e.what());
  } catch (const NotBijective& e) {
    return fail(LEGO_E_NOT_BIJECTIVE, e.what());
  } catch (const HipFailure& e) {
    return fail(LEGO_E_HIP, e.what());
  } catch (const std::length_error& e) {
    return fail(LEGO_E_SIZE_MISMATCH, e.what());
  } catch (const std::domain_error& e) {
    return fail(LEGO_E_NOT_PERMUTATION, e.what());
  } catch (const std::out_of_range& e) {
    return fail(LEGO_E_OUT_OF_RANGE, e.what());
  } catch (const std::invalid_argument& e) {
    return fail(LEGO_E_INVALID_ARG, e.what());
  } catch (const std::overflow_error& e) {
    return fail(LEGO_E_INVALID_ARG, e.what());
  } catch (const std::bad_alloc&) {
    return fail(LEGO_E_NO_MEMORY, "out of host memory");
  } catch (const std::runtime_error& e) {
    return fail(LEGO_E_JIT, e.what());
  } catch (const std::exception& e) {
    return fail(LEGO_E_INVALID_ARG, e.what());
  }
}

PieceP piece_of(lego_piece_t h) {
  if (!h || h->magic != 0x50434549u) throw std::invalid_argument("invalid piece handle");
  return h->p;
}
LayoutP layout_of(lego_layout_t h) {
  if (!h || h->magic != 0x4c41594fu) throw std::invalid_argument("invalid layout handle");
  return h->l;
}

std::vector<i64> dims_arg(int d, const int64_t* dims, int maxd = 16) {
  if (d < 1 || d > maxd) throw std::invalid_argument("rank must be in [1, " + std::to_string(maxd) + "]");
  if (!dims) throw std::invalid_argument("null dims");
  std::vector<i64> v(dims, dims + d);
  for (auto x : v)
    if (x <= 0) throw std::invalid_argument("dimension sizes must be positive");
  return v;
}

lego_status out_piece(PieceP p, lego_piece_t* out) {
  if (!out) throw std::invalid_argument("null output pointer");
  auto* h = new lego_piece_s;
  h->p = std::move(p);
  *out = h;
  return LEGO_OK;
}
lego_status out_layout(LayoutP l, lego_layout_t* out) {
  if (!out) throw std::invalid_argument("null output pointer");
  auto* h = new lego_layout_s;
  h->l = std::move(l);
  *out = h;
  return LEGO_OK;
}

void hip_check(hipError_t e, const char* what) {
  if (e != hipSuccess) throw HipFailure(std::string(what) + ": " + hipGetErrorString(e));
}

void launch(const KernelPlan& k, void** args, void* stream, long long max_wgs = 0) {
  if (k.grid <= 0 || k.grid > 0x7fffffffll) throw Unsupported("grid too large");
  int dev = 0;
  hip_check(hipGetDevice(&dev), "hipGetDevice");
  const bool slot = dev >= 0 && dev < FnCache::kDevices;
  hipFunction_t fn = nullptr;
  if (slot) {
    std::lock_guard<std::mutex> lk(k.fns.mu);
    fn = (hipFunction_t)k.fns.fn[dev];
  }
  if (!fn) {
    fn = jit_get(k.src, k.kernel).fn;
    if (slot) {
      std::lock_guard<std::mutex> lk(k.fns.mu);
      k.fns.fn[dev] = (void*)fn;
    }
  }
  long long grid = k.grid;
  if (k.persistent) {
    // A persistent kernel walks its tiles grid-stride: launch as many
    // workgroups as the device holds at once (every CU busy, no second wave
    // of workgroups), never more than there are tiles.
    long long res = 0;
    if (slot) {
      std::lock_guard<std::mutex> lk(k.fns.mu);
      res = k.fns.resident[dev];
    }
    if (!res) {
      int per_cu = 0, cus = 0;
      hip_check(hipModuleOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, k.block, 0),
                "hipModuleOccupancyMaxActiveBlocksPerMultiprocessor");
      hip_check(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev), "hipDeviceGetAttribute");
      res = (long long)std::max(1, per_cu) * std::max(1, cus);
      if (slot) {
        std::lock_guard<std::mutex> lk(k.fns.mu);
        k.fns.resident[dev] = res;
      }
    }
    grid = std::min(grid, res);
    if (max_wgs > 0) grid = std::min(grid, max_wgs);
  }
  hip_check(hipModuleLaunchKernel(fn, (unsigned)grid, 1, 1, (unsigned)k.block, 1, 1, 0, (hipStream_t)stream, args,
                                  nullptr),
            "hipModuleLaunchKernel");
}

// Plans are cached per (layout objects, parameters); the cache holds
// references, so a cached layout object is never freed and reused.
std::mutex g_plan_mu;
std::map<std::tuple<const void*, const void*, int, int>, std::pair<std::vector<LayoutP>, std::shared_ptr<KernelPlan>>>
    g_plans;

template <class Make>
std::shared_ptr<KernelPlan> cached_plan(const LayoutP& a, const LayoutP& b, int x, int y, Make make) {
  auto key = std::make_tuple((const void*)a.get(), (const void*)b.get(), x, y);
  {
    std::lock_guard<std::mutex> lk(g_plan_mu);
    auto it = g_plans.find(key);
    if (it != g_plans.end()) return it->second.second;
  }
  std::shared_ptr<KernelPlan> p = make();
  std::lock_guard<std::mutex> lk(g_plan_mu);
  g_plans[key] = {{a, b}, p};
  return p;
}

}  // namespace

extern "C" {

const char* lego_last_error(void) { return g_err.c_str(); }
const char* lego_version(void) { return "lego-mi355x 0.1 (gfx950)"; }

void lego_retain(void* handle) {
  if (!handle) return;
  uint32_t magic;
  std::memcpy(&magic, handle, sizeof magic);
  if (magic == 0x50434549u)
    ++((lego_piece_s*)handle)->rc;
  else if (magic == 0x4c41594fu)
    ++((lego_layout_s*)handle)->rc;
}

void lego_release(void* handle) {
  if (!handle) return;
  uint32_t magic;
  std::memcpy(&magic, handle, sizeof magic);
  if (magic == 0x50434549u) {
    auto* h = (lego_piece_s*)handle;
    if (--h->rc == 0) {
      h->magic = 0;
      delete h;
    }
  } else if (magic == 0x4c41594fu) {
    auto* h = (lego_layout_s*)handle;
    if (--h->rc == 0) {
      h->magic = 0;
      delete h;
    }
  }
}

lego_status lego_regp(int d, const int64_t* dims, const int32_t* sigma, lego_piece_t* out) {
  return guard([&] {
    auto n = dims_arg(d, dims);
    if (!sigma) throw std::invalid_argument("null sigma");
    return out_piece(make_regp(n, std::vector<int>(sigma, sigma + d)), out);
  });
}

lego_status lego_row(int d, const int64_t* dims, lego_piece_t* out) {
  return guard([&] { return out_piece(make_row(dims_arg(d, dims)), out); });
}

lego_status lego_col(int d, const int64_t* dims, lego_piece_t* out) {
  return guard([&] { return out_piece(make_col(dims_arg(d, dims)), out); });
}

lego_status lego_genp(int kind, int d, const int64_t* dims, const int64_t* params, int nparams, lego_piece_t* out) {
  return guard([&] {
    auto n = dims_arg(d, dims);
    if (nparams < 0 || (nparams > 0 && !params)) throw std::invalid_argument("bad params");
    return out_piece(make_genp(kind, n, std::vector<i64>(params, params + nparams)), out);
  });
}

lego_status lego_genp_expr(int d, const int64_t* dims, const char* apply_expr, const char* inv_exprs,
                           lego_piece_t* out) {
  return guard([&] {
    auto n = dims_arg(d, dims);
    if (!apply_expr || !inv_exprs) throw std::invalid_argument("null expression");
    std::vector<std::string> inv;
    std::string cur;
    for (const char* c = inv_exprs;; ++c) {
      if (*c == ';' || *c == 0) {
        inv.push_back(cur);
        cur.clear();
        if (!*c) break;
      } else {
        cur += *c;
      }
    }
    return out_piece(make_genp_expr(n, apply_expr, inv), out);
  });
}

lego_status lego_piece_dims(lego_piece_t p, int* rank, int64_t* dims) {
  return guard([&] {
    auto pc = piece_of(p);
    if (!rank || !dims) throw std::invalid_argument("null output");
    *rank = (int)pc->n.size();
    for (size_t k = 0; k < pc->n.size(); ++k) dims[k] = pc->n[k];
    return LEGO_OK;
  });
}

lego_status lego_groupby(int rank, const int64_t* dims, lego_layout_t* out) {
  return guard([&] { return out_layout(make_groupby(dims_arg(rank, dims, 64)), out); });
}

lego_status lego_orderby(lego_layout_t base, int n, const lego_piece_t* pieces, lego_layout_t* out) {
  return guard([&] {
    if (n < 1 || !pieces) throw std::invalid_argument("OrderBy needs at least one piece");
    std::vector<PieceP> ps;
    for (int k = 0; k < n; ++k) ps.push_back(piece_of(pieces[k]));
    return out_layout(make_orderby(layout_of(base), ps), out);
  });
}

lego_status lego_tileby(int q, int d, const int64_t* tiles, lego_layout_t* out) {
  return guard([&] {
    if (q < 1 || d < 1 || q * d > 64 || !tiles) throw std::invalid_argument("bad TileBy shape");
    return out_layout(make_tileby(q, d, dims_arg(q * d, tiles, 64)), out);
  });
}

lego_status lego_groupby_tiles(int q, int d, const int64_t* tiles, lego_layout_t* out) {
  return guard([&] {
    if (q < 1 || d < 1 || q * d > 64 || !tiles) throw std::invalid_argument("bad GroupBy tile shape");
    return out_layout(make_groupby(dims_arg(q * d, tiles, 64)), out);
  });
}

lego_status lego_tileorderby(int q, int d, const lego_piece_t* levels, lego_layout_t* out) {
  return guard([&] {
    if (q < 1 || !levels) throw std::invalid_argument("TileOrderBy needs at least one level");
    if (d < 1 || q * d > 64) throw std::invalid_argument("bad TileOrderBy shape");
    std::vector<PieceP> ps;
    for (int k = 0; k < q; ++k) {
      ps.push_back(piece_of(levels[k]));
      if ((int)ps.back()->n.size() != d) throw std::invalid_argument("a TileOrderBy level is not of rank d");
    }
    return out_layout(make_tileorderby(ps), out);
  });
}

lego_status lego_layout_from_piece(lego_piece_t p, lego_layout_t* out) {
  return guard([&] { return out_layout(make_from_piece(piece_of(p)), out); });
}

lego_status lego_expandby(int d, const int64_t* n, const int64_t* n_expanded, lego_layout_t g, lego_layout_t* out) {
  return guard([&] { return out_layout(make_expandby(dims_arg(d, n), dims_arg(d, n_expanded), layout_of(g)), out); });
}

lego_status lego_layout_rank(lego_layout_t l, int* rank) {
  return guard([&] {
    if (!rank) throw std::invalid_argument("null output");
    *rank = (int)layout_of(l)->dims().size();
    return LEGO_OK;
  });
}

lego_status lego_layout_dims(lego_layout_t l, int cap, int64_t* dims) {
  return guard([&] {
    auto lay = layout_of(l);
    if (!dims || cap < (int)lay->dims().size()) throw std::invalid_argument("dims buffer too small");
    for (size_t k = 0; k < lay->dims().size(); ++k) dims[k] = lay->dims()[k];
    return LEGO_OK;
  });
}

lego_status lego_layout_size(lego_layout_t l, int64_t* n) {
  return guard([&] {
    if (!n) throw std::invalid_argument("null output");
    *n = layout_of(l)->size();
    return LEGO_OK;
  });
}

lego_status lego_layout_phys_size(lego_layout_t l, int64_t* n) {
  return guard([&] {
    if (!n) throw std::invalid_argument("null output");
    *n = layout_of(l)->phys_size();
    return LEGO_OK;
  });
}

lego_status lego_apply(lego_layout_t l, const int64_t* idx, int64_t* flat) {
  return guard([&] {
    auto lay = layout_of(l);
    if (!idx || !flat) throw std::invalid_argument("null pointer");
    std::vector<i64> v(idx, idx + lay->dims().size());
    for (size_t k = 0; k < v.size(); ++k)
      if (v[k] < 0 || v[k] >= lay->dims()[k]) throw std::out_of_range("logical index out of range");
    *flat = host_apply(*lay, v);
    return LEGO_OK;
  });
}

lego_status lego_inv(lego_layout_t l, int64_t flat, int64_t* idx) {
  return guard([&] {
    auto lay = layout_of(l);
    if (!idx) throw std::invalid_argument("null pointer");
    if (flat < 0 || flat >= lay->phys_size()) throw std::out_of_range("physical index out of range");
    auto v = host_inv(*lay, flat);
    for (size_t k = 0; k < v.size(); ++k) idx[k] = v[k];
    return LEGO_OK;
  });
}

lego_status lego_verify_bijective(lego_layout_t l, int64_t max_points) {
  return guard([&] {
    auto lay = layout_of(l);
    i64 n = lay->size(), np = lay->phys_size();
    if (n > max_points) throw std::invalid_argument("layout has more points than max_points");
    std::vector<unsigned char> seen((size_t)np, 0);
    std::vector<i64> idx(lay->dims().size(), 0);
    i64 hits = 0;
    for (i64 x = 0; x < n; ++x) {
      i64 r = x;
      for (size_t k = idx.size(); k-- > 0;) {
        idx[k] = r % lay->dims()[k];
        r /= lay->dims()[k];
      }
      i64 f = host_apply(*lay, idx);
      if (f == -1 && lay->expand_inner) continue;
      if (f < 0 || f >= np) throw NotBijective("apply leaves the physical space at logical " + std::to_string(x));
      if (seen[(size_t)f]++) throw NotBijective("two logical points map to physical " + std::to_string(f));
      ++hits;
      auto back = host_inv(*lay, f);
      if (back != idx) throw NotBijective("inv(apply(x)) != x at logical " + std::to_string(x));
    }
    if (hits != np) throw NotBijective("apply is not onto the physical space");
    return LEGO_OK;
  });
}

lego_status lego_emit(lego_layout_t l, int which, char* buf, size_t cap, size_t* need) {
  return guard([&] {
    auto lay = layout_of(l);
    if (which != 0 && which != 1) throw std::invalid_argument("which must be 0 (apply) or 1 (inv)");
    Emitted e = emit_best(which == 0 ? "lego_apply" : "lego_inv", [&](Ctx& c) {
      return which == 0 ? spec_apply_flat(c, *lay) : spec_inv_flat(c, *lay);
    });
    std::ostringstream s;
    s << "// ops: " << e.ops << " (" << (e.expanded ? "expanded" : "unexpanded") << "), other variant: "
      << e.ops_other << "\n"
      << e.code;
    std::string t = s.str();
    if (need) *need = t.size() + 1;
    if (buf && cap) {
      size_t n = std::min(cap - 1, t.size());
      std::memcpy(buf, t.data(), n);
      buf[n] = 0;
    }
    return LEGO_OK;
  });
}

lego_status lego_apply_all_device(lego_layout_t l, int idx_bytes, void* d_out, void* stream) {
  return guard([&] {
    auto lay = layout_of(l);
    if (!d_out) throw std::invalid_argument("null device pointer");
    if ((uintptr_t)d_out & 15) throw std::invalid_argument("output must be 16-byte aligned");
    auto plan = cached_plan(lay, nullptr, 100, idx_bytes, [&] {
      return std::make_shared<KernelPlan>(plan_index_eval(*lay, 0, idx_bytes));
    });
    void* args[] = {&d_out};
    launch(*plan, args, stream);
    return LEGO_OK;
  });
}

lego_status lego_inv_all_device(lego_layout_t l, int idx_bytes, void* d_out, void* stream) {
  return guard([&] {
    auto lay = layout_of(l);
    if (!d_out) throw std::invalid_argument("null device pointer");
    if ((uintptr_t)d_out & 15) throw std::invalid_argument("output must be 16-byte aligned");
    auto plan = cached_plan(lay, nullptr, 101, idx_bytes, [&] {
      return std::make_shared<KernelPlan>(plan_index_eval(*lay, 1, idx_bytes));
    });
    void* args[] = {&d_out};
    launch(*plan, args, stream);
    return LEGO_OK;
  });
}

static std::shared_ptr<KernelPlan> remap_plan_cached(const LayoutP& s, const LayoutP& d, int eb) {
  return cached_plan(s, d, 200, eb, [&] { return std::make_shared<RemapPlan>(plan_remap(*s, *d, eb)); });
}

lego_status lego_remap(lego_layout_t src, lego_layout_t dst, int elem_bytes, const void* d_src, void* d_dst,
                       void* stream) {
  return guard([&] {
    auto s = layout_of(src), d = layout_of(dst);
    if (!d_src || !d_dst) throw std::invalid_argument("null device pointer");
    if (((uintptr_t)d_src | (uintptr_t)d_dst) & 15) throw std::invalid_argument("buffers must be 16-byte aligned");
    if (s->dims() != d->dims()) throw std::length_error("remap layouts have different logical shapes");
    const i64 sbytes = s->phys_size() * elem_bytes, dbytes = d->phys_size() * elem_bytes;
    if ((const char*)d_src < (char*)d_dst + dbytes && (char*)d_dst < (const char*)d_src + sbytes)
      throw std::invalid_argument("source and destination overlap");
    auto plan = remap_plan_cached(s, d, elem_bytes);
    void* a = const_cast<void*>(d_src);
    void* args[] = {&a, &d_dst};
    launch(*plan, args, stream);
    return LEGO_OK;
  });
}

lego_status lego_remap_plan(lego_layout_t src, lego_layout_t dst, int elem_bytes, int* path, int64_t* run, int* vec,
                            int64_t* tile, char* info, size_t info_cap) {
  return guard([&] {
    auto s = layout_of(src), d = layout_of(dst);
    auto plan = std::static_pointer_cast<RemapPlan>(remap_plan_cached(s, d, elem_bytes));
    if (path) *path = plan->path;
    if (run) *run = plan->run;
    if (vec) *vec = plan->vec;
    if (tile) *tile = plan->tile;
    if (info && info_cap) {
      size_t n = std::min(info_cap - 1, plan->info.size());
      std::memcpy(info, plan->info.data(), n);
      info[n] = 0;
    }
    return LEGO_OK;
  });
}

static lego_status copy_text(const std::string& t, char* buf, size_t cap, size_t* need) {
  if (need) *need = t.size() + 1;
  if (buf && cap) {
    size_t n = std::min(cap - 1, t.size());
    std::memcpy(buf, t.data(), n);
    buf[n] = 0;
  }
  return LEGO_OK;
}

lego_status lego_plan_source(int kind, lego_layout_t a, lego_layout_t b, int param, const lego_gemm_desc* desc,
                             char* buf, size_t cap, size_t* need) {
  return guard([&] {
    switch (kind) {
      case 0:
      case 1: {
        auto lay = layout_of(a);
        auto plan = cached_plan(lay, nullptr, 100 + kind, param, [&] {
          return std::make_shared<KernelPlan>(plan_index_eval(*lay, kind, param));
        });
        return copy_text(plan->src, buf, cap, need);
      }
      case 2:
        return copy_text(remap_plan_cached(layout_of(a), layout_of(b), param)->src, buf, cap, need);
      case 3: {
        if (!desc) throw std::invalid_argument("null descriptor");
        GemmRequest rq = gemm_request(*desc, [](lego_layout_t h) { return h ? layout_of(h) : LayoutP(); });
        return copy_text(gemm_plan_cached(rq)->src, buf, cap, need);
      }
    }
    throw std::invalid_argument("kind must be 0 (apply), 1 (inv), 2 (remap) or 3 (gemm)");
  });
}

lego_status lego_gemm(const lego_gemm_desc* desc, const void* d_a, const void* d_b, float* d_c, void* stream) {
  return guard([&] {
    if (!desc || !d_a || !d_b || !d_c) throw std::invalid_argument("null pointer");
    GemmRequest rq = gemm_request(*desc, [](lego_layout_t h) { return h ? layout_of(h) : LayoutP(); });
    // The operands are read with 16-byte vectors; C is written element by element.
    if (((uintptr_t)d_a | (uintptr_t)d_b) & 15) throw std::invalid_argument("A and B must be 16-byte aligned");
    if ((uintptr_t)d_c & 3) throw std::invalid_argument("C must be 4-byte aligned");
    if (rq.M > 0 && rq.N > 0 && rq.K > 0) {
      auto bytes = [](const LayoutP& l, i64 n, i64 eb) { return (l ? l->phys_size() : n) * eb; };
      const i64 ab = bytes(rq.a, rq.M * rq.K, 2), bb = bytes(rq.b, rq.K * rq.N, 2), cb = bytes(rq.c, rq.M * rq.N, 4);
      auto overlap = [](const void* x, i64 xn, const void* y, i64 yn) {
        return (const char*)x < (const char*)y + yn && (const char*)y < (const char*)x + xn;
      };
      if (overlap(d_c, cb, d_a, ab) || overlap(d_c, cb, d_b, bb)) throw std::invalid_argument("C overlaps A or B");
    }
    std::shared_ptr<GemmPlan> plan = gemm_plan_cached(rq);
    void* a = const_cast<void*>(d_a);
    void* b = const_cast<void*>(d_b);
    void* args[] = {&a, &b, &d_c};
    if (desc->max_workgroups < 0) throw std::invalid_argument("max_workgroups must not be negative");
    launch(*plan, args, stream, desc->max_workgroups);
    return LEGO_OK;
  });
}

lego_status lego_gemm_plan(const lego_gemm_desc* desc, char* info, size_t info_cap) {
  return guard([&] {
    if (!desc) throw std::invalid_argument("null pointer");
    GemmRequest rq = gemm_request(*desc, [](lego_layout_t h) { return h ? layout_of(h) : LayoutP(); });
    std::shared_ptr<GemmPlan> plan = gemm_plan_cached(rq);
    if (info && info_cap) {
      size_t n = std::min(info_cap - 1, plan->info.size());
      std::memcpy(info, plan->info.data(), n);
      info[n] = 0;
    }
    return LEGO_OK;
  });
}

lego_status lego_mfma_fragment_layout(int instr, int operand, lego_layout_t* out) {
  return guard([&] { return out_layout(mfma_fragment_layout(instr, operand), out); });
}

lego_status lego_selftest_source(int index, char* name, size_t name_cap, char* src, size_t src_cap, size_t* need) {
  return guard([&] {
    static std::vector<std::pair<std::string, std::string>> srcs = selftest_sources();
    if (index < 0 || index >= (int)srcs.size()) throw std::out_of_range("no such self-test source");
    const auto& [nm, text] = srcs[index];
    if (need) *need = text.size() + 1;
    if (name && name_cap) {
      size_t k = std::min(name_cap - 1, nm.size());
      std::memcpy(name, nm.data(), k);
      name[k] = 0;
    }
    if (src && src_cap) {
      size_t k = std::min(src_cap - 1, text.size());
      std::memcpy(src, text.data(), k);
      src[k] = 0;
    }
    return LEGO_OK;
  });
}

lego_status lego_selftest_compile(int* count, char* info, size_t info_cap) {
  return guard([&] {
    std::vector<std::pair<std::string, std::string>> srcs = selftest_sources();
    std::ostringstream s;
    s << "compiler: " << jit_compiler() << "\n";
    int n = 0;
    for (auto& [name, src] : srcs) {
      std::string log;
      double ms = 0;
      jit_compile(src, &log, &ms);
      s << name << ": " << (int)ms << " ms\n";
      ++n;
    }
    if (count) *count = n;
    std::string t = s.str();
    if (info && info_cap) {
      size_t k = std::min(info_cap - 1, t.size());
      std::memcpy(info, t.data(), k);
      info[k] = 0;
    }
    return LEGO_OK;
  });
}

}  // extern "C"
