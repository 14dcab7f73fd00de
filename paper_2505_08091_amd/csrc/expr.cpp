// Index-expression IR: canonical sums of digit fields and opaque atoms.
// See expr.hpp for the representation and the simplification rules.
#include "expr.hpp"

#include <algorithm>
#include <cstdlib>
#include <functional>
#include <stdexcept>

namespace lego {

namespace {

i64 floordiv(i64 a, i64 b) {
  i64 q = a / b;
  if ((a % b != 0) && ((a < 0) != (b < 0))) --q;
  return q;
}
i64 floormod(i64 a, i64 b) { return a - floordiv(a, b) * b; }

bool is_pow2(i64 x) { return x > 0 && (x & (x - 1)) == 0; }
int log2i(i64 x) {
  int s = 0;
  while ((i64(1) << s) < x) ++s;
  return s;
}

i64 isqrt_exact(i64 x) {
  if (x <= 0) return 0;
  // Digit-by-digit (binary restoring) square root.
  unsigned long long v = (unsigned long long)x, r = 0, bit = 1ull << 62;
  while (bit > v) bit >>= 2;
  while (bit) {
    if (v >= r + bit) {
      v -= r + bit;
      r = (r >> 1) + bit;
    } else {
      r >>= 1;
    }
    bit >>= 2;
  }
  return (i64)r;
}

Interval imul(Interval a, Interval b) {
  i64 c[4] = {a.lo * b.lo, a.lo * b.hi, a.hi * b.lo, a.hi * b.hi};
  return {*std::min_element(c, c + 4), *std::max_element(c, c + 4)};
}

std::string skey(const Sum& s);

AtomP make_field(const Ctx& c, int v, i64 a, i64 b) {
  if (a <= 0 || b < 0) throw std::logic_error("bad field");
  i64 hi = c.vars.at(v).hi;
  if (a > hi) return nullptr;
  i64 q = hi / a;
  if (b != 0 && q < b) b = 0;
  i64 rhi = b ? b - 1 : q;
  if (rhi == 0) return nullptr;
  auto at = std::make_shared<Atom>();
  at->op = Op::Field;
  at->var = v;
  at->a = a;
  at->b = b;
  at->r = {0, rhi};
  at->key = "f" + std::to_string(v) + "/" + std::to_string(a) + "%" + std::to_string(b);
  return at;
}

AtomP make_op(Op op, std::vector<Sum> kids, i64 k, Interval r) {
  auto at = std::make_shared<Atom>();
  at->op = op;
  at->kids = std::move(kids);
  at->k = k;
  at->r = r;
  static const char* names[] = {"F", "div", "mod", "mul", "xor", "lt", "sel", "isqrt"};
  std::string key = names[(int)op];
  key += "(";
  for (size_t i = 0; i < at->kids.size(); ++i) {
    if (i) key += ",";
    key += skey(at->kids[i]);
  }
  if (op == Op::Div || op == Op::Mod) key += ";" + std::to_string(k);
  key += ")";
  at->key = key;
  return at;
}

Sum atom_sum(AtomP a, i64 coeff = 1) {
  Sum s;
  if (a && coeff) s.t.push_back({coeff, a});
  return s;
}

// Sort, merge equal atoms, drop zero terms, then merge adjacent digit fields
// of one variable: c*((v/a)%b) + c*b*((v/(a*b))%b2) -> c*((v/a)%(b*b2)).
Sum canon(const Ctx& c, i64 c0, std::vector<Term> ts) {
  for (;;) {
    std::sort(ts.begin(), ts.end(), [](const Term& x, const Term& y) { return x.a->key < y.a->key; });
    std::vector<Term> m;
    for (auto& t : ts) {
      if (!m.empty() && m.back().a->key == t.a->key) {
        m.back().c += t.c;
      } else {
        m.push_back(t);
      }
    }
    ts.clear();
    for (auto& t : m)
      if (t.c != 0) ts.push_back(t);
    // field merging
    bool merged = false;
    for (size_t i = 0; i < ts.size() && !merged; ++i) {
      const Atom& f1 = *ts[i].a;
      if (f1.op != Op::Field || f1.b == 0) continue;
      for (size_t j = 0; j < ts.size(); ++j) {
        if (j == i) continue;
        const Atom& f2 = *ts[j].a;
        if (f2.op != Op::Field || f2.var != f1.var) continue;
        if (f2.a == f1.a * f1.b && ts[j].c == ts[i].c * f1.b) {
          AtomP nf = make_field(c, f1.var, f1.a, f2.b == 0 ? 0 : f1.b * f2.b);
          i64 cc = ts[i].c;
          std::vector<Term> rest;
          for (size_t k = 0; k < ts.size(); ++k)
            if (k != i && k != j) rest.push_back(ts[k]);
          if (nf) rest.push_back({cc, nf});
          ts = std::move(rest);
          merged = true;
          break;
        }
      }
    }
    if (!merged) break;
  }
  Sum s;
  s.c0 = c0;
  s.t = std::move(ts);
  return s;
}

std::string skey(const Sum& s) {
  std::string k = std::to_string(s.c0);
  for (auto& t : s.t) k += "+" + std::to_string(t.c) + "*" + t.a->key;
  return k;
}

Sum div_atom(const Ctx& c, const Sum& L, i64 n);
Sum mod_atom(const Ctx& c, const Sum& L, i64 n);

// Split x = H + L where every coefficient of H (and H.c0) is a multiple of n.
void split(const Ctx& c, const Sum& x, i64 n, Sum* H, Sum* L) {
  std::vector<Term> ht, lt;
  i64 hc0 = floordiv(x.c0, n) * n;
  i64 lc0 = x.c0 - hc0;
  for (auto& t : x.t) {
    if (t.c % n == 0) {
      ht.push_back(t);
      continue;
    }
    if (c.expand) {
      i64 ac = std::llabs(t.c);
      if (n % ac == 0) {
        i64 m = n / ac;
        const Atom& a = *t.a;
        if (a.op == Op::Field && (a.b == 0 || a.b % m == 0)) {
          AtomP lo = make_field(c, a.var, a.a, m);
          AtomP hi = make_field(c, a.var, a.a * m, a.b ? a.b / m : 0);
          if (lo) lt.push_back({t.c, lo});
          if (hi) ht.push_back({t.c * m, hi});
          continue;
        }
        if (a.op == Op::Xor && is_pow2(m) && a.kids[0].t.size() + a.kids[1].t.size() > 0 &&
            range(a.kids[0]).lo >= 0 && range(a.kids[1]).lo >= 0) {
          // Bitwise xor commutes with shifting and masking by powers of two.
          Sum lo = bxor(c, fmod(c, a.kids[0], m), fmod(c, a.kids[1], m));
          Sum hi = bxor(c, fdiv(c, a.kids[0], m), fdiv(c, a.kids[1], m));
          Sum lo2 = mulc(c, lo, t.c), hi2 = mulc(c, hi, t.c * m);
          lc0 += lo2.c0;
          hc0 += hi2.c0;
          for (auto& u : lo2.t) lt.push_back(u);
          for (auto& u : hi2.t) ht.push_back(u);
          continue;
        }
      }
    }
    lt.push_back(t);
  }
  // Constants may have moved between the parts; renormalise c0 split.
  i64 extra = floordiv(lc0, n) * n;
  hc0 += extra;
  lc0 -= extra;
  *H = canon(c, hc0, ht);
  *L = canon(c, lc0, lt);
}

Sum exact_div(const Ctx& c, const Sum& H, i64 n) {
  std::vector<Term> ts;
  for (auto& t : H.t) ts.push_back({t.c / n, t.a});
  return canon(c, H.c0 / n, ts);
}

// x = A + B with A a multiple of g (its constant and every coefficient), B in
// [0, g) and g a power of two dividing n; tries the largest such g first.
// Then (A + B) div n = A div n, (A + B) mod n = (A mod n) + B and
// A + B < n  <=>  A < n.  This is what keeps a vector of g consecutive
// positions together under a modulus that is not a power of two.
i64 gcd64(i64 a, i64 b) {
  a = a < 0 ? -a : a;
  b = b < 0 ? -b : b;
  while (b) {
    i64 t = a % b;
    a = b;
    b = t;
  }
  return a;
}
// A divisor every value of the atom is known to have.
i64 atom_multiple(const Atom& a);

}  // namespace

i64 known_multiple(const Sum& s) {
  i64 g = s.c0;
  for (const Term& t : s.t) g = gcd64(g, t.c * atom_multiple(*t.a));
  return g;
}

namespace {

i64 atom_multiple(const Atom& a) {
  switch (a.op) {
    case Op::Mod: return gcd64(known_multiple(a.kids[0]), a.k);
    case Op::Mul: return known_multiple(a.kids[0]) * known_multiple(a.kids[1]);
    case Op::Select: return gcd64(known_multiple(a.kids[1]), known_multiple(a.kids[2]));
    default: return 1;
  }
}

bool split_aligned(const Sum& x, i64 n, Sum* A, Sum* B) {
  if (n <= 1) return false;
  for (i64 g = n & -n; g >= 2; g >>= 1) {
    if (x.c0 % g) continue;
    Sum a, b;
    a.c0 = x.c0;
    for (const Term& t : x.t) ((t.c * atom_multiple(*t.a)) % g == 0 ? a : b).t.push_back(t);
    if (b.t.empty() || a.t.empty()) continue;
    Interval rb = range(b);
    if (rb.lo >= 0 && rb.hi < g) {
      *A = a;
      *B = b;
      return true;
    }
  }
  return false;
}

Sum div_atom(const Ctx& c, const Sum& L, i64 n) {
  if (L.is_const()) return cst(floordiv(L.c0, n));
  Interval r = range(L);
  if (r.lo >= 0 && r.hi < n) return cst(0);
  {
    Sum A, B;
    if (split_aligned(L, n, &A, &B)) return fdiv(c, A, n);
  }
  if (L.c0 == 0 && L.t.size() == 1 && L.t[0].c == 1) {
    const Atom& a = *L.t[0].a;
    if (a.op == Op::Div && range(a.kids[0]).lo >= 0) return div_atom(c, a.kids[0], a.k * n);
    if (a.op == Op::Field && (a.b == 0 || a.b % n == 0))
      return atom_sum(make_field(c, a.var, a.a * n, a.b ? a.b / n : 0));
  }
  return atom_sum(make_op(Op::Div, {L}, n, {floordiv(r.lo, n), floordiv(r.hi, n)}));
}

Sum mod_atom(const Ctx& c, const Sum& L, i64 n) {
  if (L.is_const()) return cst(floormod(L.c0, n));
  Interval r = range(L);
  if (r.lo >= 0 && r.hi < n) return L;
  {
    Sum A, B;
    if (split_aligned(L, n, &A, &B)) return add(c, fmod(c, A, n), B);
  }
  if (L.c0 == 0 && L.t.size() == 1 && L.t[0].c == 1) {
    const Atom& a = *L.t[0].a;
    if (a.op == Op::Field && (a.b == 0 || a.b % n == 0)) return atom_sum(make_field(c, a.var, a.a, n));
    if (a.op == Op::Mod && a.k % n == 0) return mod_atom(c, a.kids[0], n);
  }
  Interval out{0, n - 1};
  if (r.lo >= 0) out.hi = std::min(out.hi, r.hi);
  return atom_sum(make_op(Op::Mod, {L}, n, out));
}

void collect_vars(const Atom& a, std::vector<bool>& used) {
  if (a.op == Op::Field) {
    if ((int)used.size() <= a.var) used.resize(a.var + 1, false);
    used[a.var] = true;
    return;
  }
  for (auto& k : a.kids) vars_of(k, used);
}

}  // namespace

int Ctx::var(const std::string& name, i64 extent) {
  if (extent <= 0) throw std::invalid_argument("variable extent must be positive");
  vars.push_back({name, extent - 1});
  return (int)vars.size() - 1;
}

Sum cst(i64 v) {
  Sum s;
  s.c0 = v;
  return s;
}

Sum var(const Ctx& c, int v) { return field(c, v, 1, 0); }

Sum field(const Ctx& c, int v, i64 a, i64 b) { return atom_sum(make_field(c, v, a, b)); }

Sum add(const Ctx& c, const Sum& x, const Sum& y) {
  std::vector<Term> ts = x.t;
  ts.insert(ts.end(), y.t.begin(), y.t.end());
  return canon(c, x.c0 + y.c0, ts);
}

Sum mulc(const Ctx& c, const Sum& x, i64 k) {
  if (k == 0) return cst(0);
  std::vector<Term> ts;
  for (auto& t : x.t) ts.push_back({t.c * k, t.a});
  return canon(c, x.c0 * k, ts);
}

Sum sub(const Ctx& c, const Sum& x, const Sum& y) { return add(c, x, mulc(c, y, -1)); }

Sum mul(const Ctx& c, const Sum& x, const Sum& y) {
  if (x.is_const()) return mulc(c, y, x.c0);
  if (y.is_const()) return mulc(c, x, y.c0);
  std::vector<Sum> k = {x, y};
  std::sort(k.begin(), k.end(), [](const Sum& a, const Sum& b) { return skey(a) < skey(b); });
  return atom_sum(make_op(Op::Mul, k, 0, imul(range(x), range(y))));
}

Sum fdiv(const Ctx& c, const Sum& x, i64 n) {
  if (n <= 0) throw std::invalid_argument("division by a non-positive constant");
  if (n == 1) return x;
  if (x.is_const()) return cst(floordiv(x.c0, n));
  Sum H, L;
  split(c, x, n, &H, &L);
  return add(c, exact_div(c, H, n), div_atom(c, L, n));
}

Sum fmod(const Ctx& c, const Sum& x, i64 n) {
  if (n <= 0) throw std::invalid_argument("modulo by a non-positive constant");
  if (n == 1) return cst(0);
  if (x.is_const()) return cst(floormod(x.c0, n));
  Sum H, L;
  split(c, x, n, &H, &L);
  return mod_atom(c, L, n);
}

// max(x, 0), as select(x < 0, 0, x).  XOR and the integer square root are
// only defined here for non-negative operands; where the interval analysis
// cannot show that (it loses the correlation between the terms of, e.g., the
// triangle offset y - d(d+1)/2 of an antidiagonal inverse) but the operand is
// a coordinate, which is never negative for an index in range, the operand is
// clamped, a no-op on every index in range.
static Sum clamp0(const Ctx& c, const Sum& x) {
  if (range(x).lo >= 0) return x;
  return select(c, lt(c, x, cst(0)), cst(0), x);
}

Sum bxor(const Ctx& c, const Sum& x0, const Sum& y0) {
  const Sum x = clamp0(c, x0), y = clamp0(c, y0);
  if (x.is_const() && y.is_const()) return cst(x.c0 ^ y.c0);
  if (x.is_const() && x.c0 == 0) return y;
  if (y.is_const() && y.c0 == 0) return x;
  if (skey(x) == skey(y)) return cst(0);
  Interval rx = range(x), ry = range(y);
  if (rx.lo < 0 || ry.lo < 0) throw std::invalid_argument("xor of a possibly negative value");
  i64 m = std::max(rx.hi, ry.hi);
  i64 hi = 1;
  while (hi <= m) hi <<= 1;
  std::vector<Sum> k = {x, y};
  std::sort(k.begin(), k.end(), [](const Sum& a, const Sum& b) { return skey(a) < skey(b); });
  return atom_sum(make_op(Op::Xor, k, 0, {0, hi - 1}));
}

Sum lt(const Ctx& c, const Sum& x, const Sum& y) {
  Interval rx = range(x), ry = range(y);
  if (rx.hi < ry.lo) return cst(1);
  if (rx.lo >= ry.hi) return cst(0);
  // A vector of g consecutive positions shares one bounds test.
  if (y.is_const() && y.c0 > 0) {
    Sum A, B;
    if (split_aligned(x, y.c0, &A, &B)) return lt(c, A, y);
  }
  return atom_sum(make_op(Op::Lt, {x, y}, 0, {0, 1}));
}

Sum select(const Ctx& c, const Sum& cond, const Sum& x, const Sum& y) {
  if (cond.is_const()) return cond.c0 ? x : y;
  if (skey(x) == skey(y)) return x;
  // Terms both operands have, with equal coefficients, are added outside:
  // c ? X + t : Y + t = t + (c ? X : Y).  (A term of a variable common to
  // both branches then stays out of the select, so a sum can still be split
  // by that variable.)
  Sum common, xr, yr;
  xr.c0 = x.c0;
  yr.c0 = y.c0;
  size_t i = 0, j = 0;
  while (i < x.t.size() || j < y.t.size()) {
    const int cmp = i == x.t.size() ? 1 : j == y.t.size() ? -1 : x.t[i].a->key.compare(y.t[j].a->key);
    if (cmp < 0) {
      xr.t.push_back(x.t[i++]);
    } else if (cmp > 0) {
      yr.t.push_back(y.t[j++]);
    } else {
      if (x.t[i].c == y.t[j].c) {
        common.t.push_back(x.t[i]);
      } else {
        xr.t.push_back(x.t[i]);
        yr.t.push_back(y.t[j]);
      }
      ++i;
      ++j;
    }
  }
  if (!common.t.empty()) return add(c, common, select(c, cond, xr, yr));
  Interval rx = range(x), ry = range(y);
  Interval r{std::min(rx.lo, ry.lo), std::max(rx.hi, ry.hi)};
  // select(y < 0, 0, y) is max(y, 0): never negative
  if (x.is_const() && x.c0 == 0 && cond.c0 == 0 && cond.t.size() == 1 && cond.t[0].c == 1 &&
      cond.t[0].a->op == Op::Lt && cond.t[0].a->kids[1].is_const() && cond.t[0].a->kids[1].c0 == 0 &&
      skey(cond.t[0].a->kids[0]) == skey(y))
    r.lo = std::max<i64>(r.lo, 0);
  return atom_sum(make_op(Op::Select, {cond, x, y}, 0, r));
}

Sum isqrt(const Ctx& c, const Sum& x0) {
  const Sum x = clamp0(c, x0);
  if (x.is_const()) return cst(isqrt_exact(x.c0));
  Interval r = range(x);
  if (r.lo < 0) throw std::invalid_argument("isqrt of a possibly negative value");
  return atom_sum(make_op(Op::Isqrt, {x}, 0, {isqrt_exact(r.lo), isqrt_exact(r.hi)}));
}

Interval range(const Sum& s) {
  Interval r{s.c0, s.c0};
  for (auto& t : s.t) {
    if (t.c > 0) {
      r.lo += t.c * t.a->r.lo;
      r.hi += t.c * t.a->r.hi;
    } else {
      r.lo += t.c * t.a->r.hi;
      r.hi += t.c * t.a->r.lo;
    }
  }
  return r;
}

std::string key(const Sum& s) { return skey(s); }

void vars_of(const Sum& s, std::vector<bool>& used) {
  for (auto& t : s.t) collect_vars(*t.a, used);
}

bool depends_on(const Sum& s, int v) {
  std::vector<bool> u;
  vars_of(s, u);
  return v < (int)u.size() && u[v];
}

Sum subst(const Ctx& c, const Sum& s, int v, const Sum& repl) {
  std::map<std::string, Sum> memo;
  std::function<Sum(const Sum&)> go_sum;
  std::function<Sum(const Atom&)> go_atom = [&](const Atom& a) -> Sum {
    auto it = memo.find(a.key);
    if (it != memo.end()) return it->second;
    Sum r;
    switch (a.op) {
      case Op::Field:
        if (a.var != v) {
          r = field(c, a.var, a.a, a.b);
        } else {
          r = fdiv(c, repl, a.a);
          if (a.b) r = fmod(c, r, a.b);
        }
        break;
      case Op::Div: r = fdiv(c, go_sum(a.kids[0]), a.k); break;
      case Op::Mod: r = fmod(c, go_sum(a.kids[0]), a.k); break;
      case Op::Mul: r = mul(c, go_sum(a.kids[0]), go_sum(a.kids[1])); break;
      case Op::Xor: r = bxor(c, go_sum(a.kids[0]), go_sum(a.kids[1])); break;
      case Op::Lt: r = lt(c, go_sum(a.kids[0]), go_sum(a.kids[1])); break;
      case Op::Select: r = select(c, go_sum(a.kids[0]), go_sum(a.kids[1]), go_sum(a.kids[2])); break;
      case Op::Isqrt: r = isqrt(c, go_sum(a.kids[0])); break;
    }
    memo[a.key] = r;
    return r;
  };
  go_sum = [&](const Sum& x) -> Sum {
    Sum out = cst(x.c0);
    for (auto& t : x.t) out = add(c, out, mulc(c, go_atom(*t.a), t.c));
    return out;
  };
  return go_sum(s);
}

bool split_by(const Sum& s, const std::vector<int>& group, Sum* in_group, Sum* rest) {
  Sum a, b;
  b.c0 = s.c0;
  for (auto& t : s.t) {
    std::vector<bool> u;
    collect_vars(*t.a, u);
    bool any_in = false, any_out = false;
    for (int v = 0; v < (int)u.size(); ++v) {
      if (!u[v]) continue;
      bool in = std::find(group.begin(), group.end(), v) != group.end();
      (in ? any_in : any_out) = true;
    }
    if (any_in && any_out) return false;
    (any_in ? a : b).t.push_back(t);
  }
  *in_group = a;
  *rest = b;
  return true;
}

bool digits_of(const Ctx& c, const Sum& s, int v, std::vector<Digit>* out) {
  out->clear();
  // A digit permutation has no constant and positive digit weights (a map
  // such as n - 1 - p, a reversal, is a bijection but not of this form).
  if (s.c0 != 0) return false;
  for (auto& t : s.t) {
    const Atom& a = *t.a;
    if (a.op != Op::Field || a.var != v || t.c <= 0) return false;
    i64 b = a.b ? a.b : (c.vars[v].hi / a.a + 1);
    out->push_back({a.a, b, t.c});
  }
  std::sort(out->begin(), out->end(), [](const Digit& x, const Digit& y) { return x.a < y.a; });
  i64 next = 1;
  for (auto& d : *out) {
    if (d.a != next) return false;
    next = d.a * d.b;
  }
  return next == c.vars[v].hi + 1;
}

// ------------------------------------------------------------------ print --
namespace {

// 32-bit index code computes sums, products and selects modulo 2^32, which
// gives the true value wherever that value lies in [0, 2^32) whatever the
// intermediate values were; the other operations (floor division, modulo,
// comparison, xor, square root, a select's condition) need their operands'
// true values, so those must be proven in [0, 2^32) by their ranges.
bool sum_fits32(const Sum& s);

// The 32-bit evaluation of `s` is congruent to its value modulo 2^32.
bool sum_ring32(const Sum& s);

bool atom_ring32(const Atom& a) {
  switch (a.op) {
    case Op::Mul:
      return sum_ring32(a.kids[0]) && sum_ring32(a.kids[1]);
    case Op::Select:
      return sum_fits32(a.kids[0]) && sum_ring32(a.kids[1]) && sum_ring32(a.kids[2]);
    default:
      for (auto& k : a.kids)
        if (!sum_fits32(k)) return false;
      return a.r.lo >= 0 && a.r.hi < (i64(1) << 32);
  }
}

bool sum_ring32(const Sum& s) {
  for (auto& t : s.t)
    if (!atom_ring32(*t.a)) return false;
  return true;
}

// The 32-bit evaluation of `s` is its value.
bool sum_fits32(const Sum& s) {
  Interval r = range(s);
  if (r.lo < 0 || r.hi >= (i64(1) << 32)) return false;
  return sum_ring32(s);
}

struct Printer {
  const Ctx& c;
  bool wide;
  int ops = 0;
  // Common-subexpression sharing: an opaque atom referenced more than once is
  // bound to a local constant the first time it is printed.
  std::map<std::string, int> uses;
  std::map<std::string, std::string> names;
  std::vector<std::string> lets;

  void count(const Sum& s) {
    for (auto& t : s.t) count_atom(*t.a);
  }
  void count_atom(const Atom& a) {
    if (a.op == Op::Field) return;
    if (uses[a.key]++ == 0)
      for (auto& k : a.kids) count(k);
  }

  std::string lit(i64 v) {
    if (wide) return std::to_string(v) + "ll";
    return std::to_string(v) + "u";
  }

  std::string atom(const Atom& a) {
    if (a.op != Op::Field && uses[a.key] > 1) {
      auto it = names.find(a.key);
      if (it != names.end()) return it->second;
      std::string body = atom_body(a);
      std::string nm = "t" + std::to_string(lets.size());
      lets.push_back(std::string("const ") + (wide ? "i64 " : "u32 ") + nm + " = " + body + ";");
      names[a.key] = nm;
      return nm;
    }
    return atom_body(a);
  }

  std::string atom_body(const Atom& a) {
    switch (a.op) {
      case Op::Field: {
        std::string s = c.vars[a.var].name;
        if (a.a != 1) {
          ++ops;
          s = is_pow2(a.a) ? "(" + s + " >> " + std::to_string(log2i(a.a)) + ")"
                           : "(" + s + " / " + lit(a.a) + ")";
        }
        if (a.b) {
          ++ops;
          s = is_pow2(a.b) ? "(" + s + " & " + lit(a.b - 1) + ")" : "(" + s + " % " + lit(a.b) + ")";
        }
        return s;
      }
      case Op::Div: {
        ++ops;
        std::string k = sum(a.kids[0]);
        if (range(a.kids[0]).lo < 0) return "lego_fdiv(" + k + ", " + lit(a.k) + ")";
        return is_pow2(a.k) ? "(" + k + " >> " + std::to_string(log2i(a.k)) + ")" : "(" + k + " / " + lit(a.k) + ")";
      }
      case Op::Mod: {
        ++ops;
        std::string k = sum(a.kids[0]);
        if (range(a.kids[0]).lo < 0) return "lego_fmod(" + k + ", " + lit(a.k) + ")";
        return is_pow2(a.k) ? "(" + k + " & " + lit(a.k - 1) + ")" : "(" + k + " % " + lit(a.k) + ")";
      }
      case Op::Mul: ++ops; return "(" + sum(a.kids[0]) + " * " + sum(a.kids[1]) + ")";
      case Op::Xor: ++ops; return "(" + sum(a.kids[0]) + " ^ " + sum(a.kids[1]) + ")";
      case Op::Lt: ++ops; return "(" + sum(a.kids[0]) + " < " + sum(a.kids[1]) + " ? " + lit(1) + " : " + lit(0) + ")";
      case Op::Select:
        ops += 1;
        return "(" + sum(a.kids[0]) + " ? " + sum(a.kids[1]) + " : " + sum(a.kids[2]) + ")";
      case Op::Isqrt: ops += 12; return "lego_isqrt(" + sum(a.kids[0]) + ")";
    }
    return "?";
  }

  std::string term(const Term& t, bool neg) {
    i64 c0 = neg ? -t.c : t.c;
    std::string a = atom(*t.a);
    if (c0 == 1) return a;
    ++ops;
    if (is_pow2(c0)) return "(" + a + " << " + std::to_string(log2i(c0)) + ")";
    return "(" + a + " * " + lit(c0) + ")";
  }

  std::string sum(const Sum& s) {
    std::string out;
    int n = 0;
    for (auto& t : s.t) {
      if (t.c < 0) continue;
      if (n++) {
        out += " + ";
        ++ops;
      }
      out += term(t, false);
    }
    for (auto& t : s.t) {
      if (t.c > 0) continue;
      if (n++) {
        out += " - ";
        ++ops;
        out += term(t, true);
      } else {
        ++ops;
        out += "(" + lit(0) + " - " + term(t, true) + ")";
      }
    }
    if (s.c0 != 0 || n == 0) {
      if (n) {
        ++ops;
        out += s.c0 < 0 ? " - " + lit(-s.c0) : " + " + lit(s.c0);
      } else {
        out += s.c0 < 0 ? "(" + lit(0) + " - " + lit(-s.c0) + ")" : lit(s.c0);
      }
    }
    return n + (s.c0 != 0) > 1 ? "(" + out + ")" : out;
  }
};

}  // namespace

bool fits32(const Sum& s) { return sum_fits32(s); }
bool ring32(const Sum& s) { return sum_ring32(s); }

Printed print(const Ctx& c, const Sum& s) {
  PrintedMany m = print_many(c, {s}, !sum_fits32(s));
  Printed out;
  out.text = m.lets.empty() ? m.outs[0] : "({ " + m.lets + " " + m.outs[0] + "; })";
  out.ops = m.ops;
  out.wide = !sum_fits32(s);
  return out;
}

PrintedMany print_many(const Ctx& c, const std::vector<Sum>& outs, bool wide) {
  Printer p{c, wide};
  for (auto& s : outs) p.count(s);
  PrintedMany m;
  for (auto& s : outs) m.outs.push_back(p.sum(s));
  for (auto& l : p.lets) m.lets += l + "\n";
  m.ops = p.ops;
  return m;
}

}  // namespace lego
