// Lowering layouts to straight-line index code.  See lower.hpp.
#include "lower.hpp"

#include <sstream>
#include <stdexcept>

namespace lego {

std::string fn_text(const Ctx& c, const std::string& name, const FnSpec& f, bool force_wide, int* ops,
                    bool* wide) {
  bool w = force_wide;
  for (size_t k = 0; k < f.outs.size(); ++k) {
    const bool bounded = k < f.out_bound.size() && f.out_bound[k] > 0 && f.out_bound[k] <= (i64(1) << 32);
    w = w || !(bounded || f.ring_out ? ring32(f.outs[k]) : fits32(f.outs[k]));
  }
  for (int v : f.params) w = w || c.vars[v].hi >= (i64(1) << 32);
  const char* T = w ? "i64" : "u32";
  std::ostringstream s;
  int n = 0;
  if (f.outs.size() == 1 && !f.out_array) {
    s << "LEGO_FN " << T << " " << name << "(";
  } else {
    s << "LEGO_FN void " << name << "(";
  }
  for (size_t k = 0; k < f.params.size(); ++k) s << (k ? ", " : "") << T << " " << c.vars[f.params[k]].name;
  if (f.out_array) {
    s << (f.params.empty() ? "" : ", ") << T << "* __restrict__ o";
  } else if (f.outs.size() != 1) {
    for (size_t k = 0; k < f.outs.size(); ++k)
      s << (f.params.empty() && k == 0 ? "" : ", ") << T << "* __restrict__ o" << k;
  }
  s << ") {\n";
  PrintedMany pm = print_many(c, f.outs, w);
  n = pm.ops;
  if (!pm.lets.empty()) {
    std::istringstream ls(pm.lets);
    std::string line;
    while (std::getline(ls, line)) s << "  " << line << "\n";
  }
  for (size_t k = 0; k < f.outs.size(); ++k) {
    if (f.out_array)
      s << "  o[" << k << "] = " << pm.outs[k] << ";\n";
    else if (f.outs.size() == 1)
      s << "  return " << pm.outs[k] << ";\n";
    else
      s << "  *o" << k << " = " << pm.outs[k] << ";\n";
  }
  s << "}\n";
  if (ops) *ops = n;
  if (wide) *wide = w;
  return s.str();
}

Emitted emit_best(const std::string& name, const std::function<FnSpec(Ctx&)>& build, bool force_wide, int variant) {
  Emitted best;
  int ops[2] = {0, 0};
  std::string text[2];
  bool wide[2] = {false, false}, ok[2] = {false, false};
  for (int e = 0; e < 2; ++e) {
    if (variant >= 0 && e != variant) continue;
    Ctx c;
    c.expand = (e == 0);
    FnSpec f = build(c);
    if (!f.valid) continue;
    ok[e] = true;
    text[e] = fn_text(c, name, f, force_wide, &ops[e], &wide[e]);
  }
  if (!ok[0] && !ok[1]) throw std::logic_error("no lowering variant can express " + name);
  int pick = !ok[1] ? 0 : !ok[0] ? 1 : (ops[0] <= ops[1] ? 0 : 1);
  best.code = text[pick];
  best.ops = ops[pick];
  best.ops_other = ok[1 - pick] ? ops[1 - pick] : -1;
  best.expanded = (pick == 0);
  best.wide = wide[pick];
  return best;
}

FnSpec spec_apply_flat(Ctx& c, const Layout& l) {
  SymAlg al{&c};
  int x = c.var("x", l.size());
  std::vector<Sum> idx = unflatten(al, l.dims(), var(c, x));
  FnSpec f;
  f.params = {x};
  f.outs = {l.apply(al, idx)};
  // a bijection onto [0, phys_size) (ExpandBy's apply is -1 off its extents)
  if (!l.expand_inner) f.out_bound = {l.phys_size()};
  return f;
}

FnSpec spec_inv_flat(Ctx& c, const Layout& l) {
  SymAlg al{&c};
  int p = c.var("p", l.phys_size());
  FnSpec f;
  f.params = {p};
  f.outs = l.inv(al, var(c, p));
  if (!l.expand_inner) f.out_bound = l.dims();
  return f;
}

Sum remap_map(Ctx& c, const Layout& src, const Layout& dst, int p) {
  SymAlg al{&c};
  return src.apply(al, dst.inv(al, var(c, p)));
}

Sum remap_map_masked(Ctx& c, const Layout& src, const Layout& dst, int p, Sum* valid) {
  SymAlg al{&c};
  std::vector<Sum> x = dst.inv(al, var(c, p));
  if (!src.expand_inner) {
    *valid = cst(1);
    return src.apply(al, x);
  }
  // ExpandBy apply (Figure 9) with its two outcomes kept apart: the point in
  // the original extents, and whether it lies inside them.
  std::vector<Sum> ip = unflatten(al, src.ne, src.expand_inner->apply(al, x));
  Sum ok = cst(1);
  for (size_t k = 0; k < src.en.size(); ++k) ok = al.mul(ok, al.lt(ip[k], al.c(src.en[k])));
  *valid = ok;
  return flatten(al, src.en, ip);
}

const char* prelude_text() {
  return R"PRELUDE(
typedef unsigned int u32;
typedef long long i64;
typedef unsigned long long u64;
#ifndef LEGO_FN
#define LEGO_FN __device__ __forceinline__
#endif
// Floor division / modulo for operands that may be negative.
LEGO_FN i64 lego_fdiv(i64 x, i64 n) { i64 q = x / n; return q - (((x % n) != 0) & ((x < 0) != (n < 0))); }
LEGO_FN i64 lego_fmod(i64 x, i64 n) { return x - lego_fdiv(x, n) * n; }
// Exact integer square root, binary digit-by-digit (restoring) method.
LEGO_FN u64 lego_isqrt_u64(u64 v) {
  u64 r = 0, bit = 1ull << 62;
  while (bit > v) bit >>= 2;
  while (bit) {
    if (v >= r + bit) { v -= r + bit; r = (r >> 1) + bit; } else { r >>= 1; }
    bit >>= 2;
  }
  return r;
}
// 32-bit operands: the square root of the nearest float, corrected to the
// exact floor by integer comparisons (the estimate is off by at most one for
// every 32-bit v; the loops make the result exact whatever the estimate).  The
// floor is at most 65535, so clamping the estimate there keeps every square
// in 32 bits.
LEGO_FN u32 lego_isqrt(u32 v) {
  u32 r = (u32)__builtin_sqrtf((float)v);
  r = r < 65535u ? r : 65535u;
  while (r * r > v) --r;
  while (r < 65535u && (r + 1) * (r + 1) <= v) ++r;
  return r;
}
LEGO_FN i64 lego_isqrt(i64 v) { return v <= 0 ? 0 : (i64)lego_isqrt_u64((u64)v); }
)PRELUDE";
}

}  // namespace lego
