// LEGO layout front end: RegP / GenP permutations, OrderBy, GroupBy chains and
// ExpandBy, with apply / inv / dims as defined in Section III-B (grammar in
// Figure 3, semantics in Figures 4 and 5) and Section III-D (Figure 9).
//
// Everything is written once, generically over an "algebra" A that supplies
// the integer operations.  IntAlg evaluates on int64 values (host apply/inv);
// SymAlg builds index expressions (expr.hpp), which is how a layout is lowered
// to kernel code: the paper evaluates its algebra on SymPy symbols in the same
// way (Section IV-A).
#pragma once

#include <memory>
#include <stdexcept>
#include <string>
#include <vector>

#include "expr.hpp"
#include "genexpr.hpp"

namespace lego {

// ----------------------------------------------------------------- algebras
struct IntAlg {
  using V = i64;
  static i64 fdiv_(i64 a, i64 b) {
    i64 q = a / b;
    if ((a % b != 0) && ((a < 0) != (b < 0))) --q;
    return q;
  }
  V c(i64 k) const { return k; }
  V add(V a, V b) const { return a + b; }
  V sub(V a, V b) const { return a - b; }
  V mulc(V a, i64 k) const { return a * k; }
  V mul(V a, V b) const { return a * b; }
  V div(V a, i64 n) const { return fdiv_(a, n); }
  V mod(V a, i64 n) const { return a - fdiv_(a, n) * n; }
  V bxor(V a, V b) const { return a ^ b; }
  V lt(V a, V b) const { return a < b ? 1 : 0; }
  V sel(V c, V a, V b) const { return c ? a : b; }
  V isqrt(V x) const;
};

struct SymAlg {
  using V = Sum;
  const Ctx* ctx;
  V c(i64 k) const { return cst(k); }
  V add(const V& a, const V& b) const { return lego::add(*ctx, a, b); }
  V sub(const V& a, const V& b) const { return lego::sub(*ctx, a, b); }
  V mulc(const V& a, i64 k) const { return lego::mulc(*ctx, a, k); }
  V mul(const V& a, const V& b) const { return lego::mul(*ctx, a, b); }
  V div(const V& a, i64 n) const { return lego::fdiv(*ctx, a, n); }
  V mod(const V& a, i64 n) const { return lego::fmod(*ctx, a, n); }
  V bxor(const V& a, const V& b) const { return lego::bxor(*ctx, a, b); }
  V lt(const V& a, const V& b) const { return lego::lt(*ctx, a, b); }
  V sel(const V& c, const V& a, const V& b) const { return lego::select(*ctx, c, a, b); }
  V isqrt(const V& x) const { return lego::isqrt(*ctx, x); }
};

// ------------------------------------------------------ canonical bijections
// B_n (Figure 4): Horner flattening, last dimension fastest.
template <class A>
typename A::V flatten(const A& al, const std::vector<i64>& n, const std::vector<typename A::V>& i) {
  typename A::V f = al.c(0);
  for (size_t k = 0; k < n.size(); ++k) f = al.add(al.mulc(f, n[k]), i[k]);
  return f;
}

// B^{-1}_n (Figure 4): repeated div/mod, last dimension fastest.
template <class A>
std::vector<typename A::V> unflatten(const A& al, const std::vector<i64>& n, typename A::V x) {
  std::vector<typename A::V> out(n.size(), al.c(0));
  for (size_t k = n.size(); k-- > 1;) {
    out[k] = al.mod(x, n[k]);
    x = al.div(x, n[k]);
  }
  if (!n.empty()) out[0] = x;
  return out;
}

template <class T>
std::vector<T> gather(const std::vector<int>& sigma, const std::vector<T>& v) {
  std::vector<T> o;
  o.reserve(sigma.size());
  for (int s : sigma) o.push_back(v[s - 1]);
  return o;
}

std::vector<int> sigma_inverse(const std::vector<int>& sigma);
std::vector<int> sigma_dq(int d, int q);
i64 product(const std::vector<i64>& v);

// ------------------------------------------------------------- permutations
enum GenKind { GEN_MORTON = 1, GEN_XOR_SWIZZLE = 2, GEN_REVERSE = 3, GEN_ANTIDIAG = 4, GEN_EXPR = 5 };

struct Piece {
  bool regp = true;
  std::vector<i64> n;      // logical dims (Figure 4 dims())
  std::vector<int> sigma;  // RegP: 1-based gather permutation
  int gk = 0;              // GenP kind
  std::vector<i64> prm;    // GenP parameters
  std::shared_ptr<const GenExpr> ex;  // GEN_EXPR: the forward and inverse expressions

  i64 size() const { return product(n); }
  std::string describe() const;

  // Figure 4: RegP apply = B_{sigma(n)}(sigma(i)); GenP apply = f(i).
  template <class A>
  typename A::V apply(const A& al, const std::vector<typename A::V>& i) const {
    if (regp) return flatten(al, gather(sigma, n), gather(sigma, i));
    return genp_apply(al, i);
  }
  // Figure 4: RegP inv = sigma^{-1}(B^{-1}_{sigma(n)}(x)); GenP inv = f^{-1}(x).
  template <class A>
  std::vector<typename A::V> inv(const A& al, const typename A::V& x) const {
    if (regp) return gather(sigma_inverse(sigma), unflatten(al, gather(sigma, n), x));
    return genp_inv(al, x);
  }

 private:
  template <class A>
  typename A::V genp_apply(const A& al, const std::vector<typename A::V>& i) const;
  template <class A>
  std::vector<typename A::V> genp_inv(const A& al, const typename A::V& x) const;
};

using PieceP = std::shared_ptr<const Piece>;

struct OrderBy {
  std::vector<PieceP> p;
  std::vector<i64> dims() const {
    std::vector<i64> d;
    for (auto& x : p) d.insert(d.end(), x->n.begin(), x->n.end());
    return d;
  }
  i64 size() const { return product(dims()); }

  // Figure 4 apply: outermost piece first, flat = piece.apply(slice) + flat*|piece|.
  template <class A>
  typename A::V apply(const A& al, const std::vector<typename A::V>& i) const {
    typename A::V flat = al.c(0);
    size_t pos = 0;
    for (auto& x : p) {
      std::vector<typename A::V> cur(i.begin() + pos, i.begin() + pos + x->n.size());
      flat = al.add(x->apply(al, cur), al.mulc(flat, x->size()));
      pos += x->n.size();
    }
    return flat;
  }
  // Figure 4 inv: innermost piece first, peel x % |piece| and prepend its inverse.
  template <class A>
  std::vector<typename A::V> inv(const A& al, typename A::V x) const {
    std::vector<typename A::V> out;
    for (size_t k = p.size(); k-- > 0;) {
      i64 sz = p[k]->size();
      typename A::V cur = al.mod(x, sz);
      x = al.div(x, sz);
      std::vector<typename A::V> sub = p[k]->inv(al, cur);
      out.insert(out.begin(), sub.begin(), sub.end());
    }
    return out;
  }
};

struct Layout;
using LayoutP = std::shared_ptr<const Layout>;

// GroupBy(tiles).OrderBy(...)... in dot notation: `chain` is in application
// order.  `g` is the concatenation of the GroupBy tile levels (the logical
// index).  An ExpandBy layout (Figure 9) wraps an inner layout over the padded
// shape `ne` and exposes the original extents `en`.
struct Layout {
  std::vector<i64> g;
  std::vector<OrderBy> chain;
  LayoutP expand_inner;  // non-null: ExpandBy(en, ne, inner)
  std::vector<i64> en, ne;

  const std::vector<i64>& dims() const { return expand_inner ? expand_inner->g : g; }
  i64 size() const { return product(dims()); }
  // Number of physical positions (differs from size() only for ExpandBy).
  i64 phys_size() const { return expand_inner ? product(en) : size(); }

  // Figure 5 apply: flatten in the logical view, then for each OrderBy in
  // application order unflatten over its dims and apply it.
  template <class A>
  typename A::V apply(const A& al, const std::vector<typename A::V>& i) const {
    if (expand_inner) {
      // Figure 9: apply through the inner layout in the expanded space; keep the
      // point only if it lies inside the original extents, else -1.
      typename A::V flat = expand_inner->apply(al, i);
      std::vector<typename A::V> ip = unflatten(al, ne, flat);
      typename A::V inside = al.c(1);
      for (size_t k = 0; k < en.size(); ++k) inside = al.mul(inside, al.lt(ip[k], al.c(en[k])));
      return al.sel(inside, flatten(al, en, ip), al.c(-1));
    }
    // When the first OrderBy has exactly the logical dims, unflatten(flatten(i))
    // is i itself: the piece then takes the coordinates directly, which keeps
    // the lowered expression linear in them (and meaningful past the extents,
    // as padded tiles need).
    size_t k0 = 0;
    typename A::V flat;
    if (!chain.empty() && chain[0].dims() == g) {
      flat = chain[0].apply(al, i);
      k0 = 1;
    } else {
      flat = flatten(al, g, i);
    }
    for (size_t k = k0; k < chain.size(); ++k) flat = chain[k].apply(al, unflatten(al, chain[k].dims(), flat));
    return flat;
  }
  // Figure 5 inv: reverse application order, O.inv then flatten over O.dims;
  // finally unflatten in the logical view.
  template <class A>
  std::vector<typename A::V> inv(const A& al, typename A::V x) const {
    if (expand_inner) {
      std::vector<typename A::V> i = unflatten(al, en, x);
      return expand_inner->inv(al, flatten(al, ne, i));
    }
    const bool direct0 = !chain.empty() && chain[0].dims() == g;
    for (size_t k = chain.size(); k-- > (direct0 ? 1 : 0);) x = flatten(al, chain[k].dims(), chain[k].inv(al, x));
    if (direct0) return chain[0].inv(al, x);
    return unflatten(al, g, x);
  }
};

// ----------------------------------------------------------- constructors
PieceP make_regp(const std::vector<i64>& n, const std::vector<int>& sigma);
PieceP make_row(const std::vector<i64>& n);
PieceP make_col(const std::vector<i64>& n);
PieceP make_genp(int kind, const std::vector<i64>& n, const std::vector<i64>& prm);
// GenP from expression text (grammar in genexpr.hpp): the forward map over
// i0..i{d-1} and one inverse expression per dimension over x.  Tiles of at most
// 2^20 points are checked exhaustively (NotBijective on failure).
PieceP make_genp_expr(const std::vector<i64>& n, const std::string& apply, const std::vector<std::string>& inv);
LayoutP make_groupby(const std::vector<i64>& dims);
LayoutP make_orderby(const LayoutP& base, const std::vector<PieceP>& pieces);
LayoutP make_tileby(int q, int d, const std::vector<i64>& tiles);
LayoutP make_tileorderby(const std::vector<PieceP>& levels);
LayoutP make_from_piece(const PieceP& p);
LayoutP make_expandby(const std::vector<i64>& en, const std::vector<i64>& ne, const LayoutP& inner);

// Host evaluation.
i64 host_apply(const Layout& l, const std::vector<i64>& idx);
std::vector<i64> host_inv(const Layout& l, i64 x);

// ----------------------------------------------------- GenP definitions
int ilog2_exact(i64 x);  // -1 if not a power of two

template <class A>
typename A::V Piece::genp_apply(const A& al, const std::vector<typename A::V>& i) const {
  using V = typename A::V;
  switch (gk) {
    case GEN_MORTON: {
      // Z order: column bits at even, row bits at odd positions while both remain.
      int br = ilog2_exact(n[0]), bc = ilog2_exact(n[1]);
      V z = al.c(0);
      int pos = 0;
      for (int b = 0; b < std::max(br, bc); ++b) {
        if (b < bc) z = al.add(z, al.mulc(al.mod(al.div(i[1], i64(1) << b), 2), i64(1) << pos++));
        if (b < br) z = al.add(z, al.mulc(al.mod(al.div(i[0], i64(1) << b), 2), i64(1) << pos++));
      }
      return z;
    }
    case GEN_XOR_SWIZZLE: {
      // f(r, c) = r*C + ((c/v) ^ ((r/s) % (C/v)))*v + c%v.
      i64 C = n[1], v = prm[0], s = prm[1];
      V hi = al.bxor(al.div(i[1], v), al.mod(al.div(i[0], s), C / v));
      return al.add(al.add(al.mulc(i[0], C), al.mulc(hi, v)), al.mod(i[1], v));
    }
    case GEN_REVERSE: {
      // Every coordinate reversed: (n1-1-i1, ..., nd-1-id) flattened.
      std::vector<V> r;
      for (size_t k = 0; k < n.size(); ++k) r.push_back(al.sub(al.c(n[k] - 1), i[k]));
      return flatten(al, n, r);
    }
    case GEN_EXPR:
      // Taken modulo the tile size: the identity on a bijection onto
      // [0, size), and it tells the lowering the range of the result.
      return al.mod(eval_gexpr(al, *ex->apply, i), size());
    case GEN_ANTIDIAG: {
      // Figure 7's order: the antidiagonals d = i + j in turn, rows
      // increasing within one.  On the upper triangle (d < n) the points
      // before (i, j) are the d(d+1)/2 of the earlier antidiagonals and the i
      // above it on its own; the lower triangle is the upper one turned by
      // 180 degrees: n*n - 1 minus the number of the turned point
      // (n-1-i, n-1-j), which lies on antidiagonal 2n-2-d.
      i64 nn = n[0];
      V d = al.add(i[0], i[1]);
      V up = al.add(al.div(al.mul(d, al.add(d, al.c(1))), 2), i[0]);
      V e = al.sub(al.c(2 * nn - 2), d);
      V turned = al.add(al.div(al.mul(e, al.add(e, al.c(1))), 2), al.sub(al.c(nn - 1), i[0]));
      return al.sel(al.lt(d, al.c(nn)), up, al.sub(al.c(nn * nn - 1), turned));
    }
  }
  throw std::logic_error("unknown GenP");
}

template <class A>
std::vector<typename A::V> Piece::genp_inv(const A& al, const typename A::V& x) const {
  using V = typename A::V;
  switch (gk) {
    case GEN_MORTON: {
      int br = ilog2_exact(n[0]), bc = ilog2_exact(n[1]);
      V r = al.c(0), c = al.c(0);
      int pos = 0;
      for (int b = 0; b < std::max(br, bc); ++b) {
        if (b < bc) c = al.add(c, al.mulc(al.mod(al.div(x, i64(1) << pos++), 2), i64(1) << b));
        if (b < br) r = al.add(r, al.mulc(al.mod(al.div(x, i64(1) << pos++), 2), i64(1) << b));
      }
      return {r, c};
    }
    case GEN_XOR_SWIZZLE: {
      i64 C = n[1], v = prm[0], s = prm[1];
      V r = al.div(x, C);
      V rest = al.mod(x, C);
      V c = al.add(al.mulc(al.bxor(al.div(rest, v), al.mod(al.div(r, s), C / v)), v), al.mod(rest, v));
      return {r, c};
    }
    case GEN_REVERSE: {
      std::vector<V> r = unflatten(al, n, al.sub(al.c(product(n) - 1), x));
      return r;
    }
    case GEN_EXPR: {
      std::vector<V> out;
      for (size_t k = 0; k < ex->inv.size(); ++k) out.push_back(al.mod(eval_gexpr(al, *ex->inv[k], std::vector<V>{x}), n[k]));
      return out;
    }
    case GEN_ANTIDIAG: {
      // Figure 7 inverse with the exact integer square root.  In the upper
      // triangle y = d(d+1)/2 + i with 0 <= i <= d on antidiagonal d, so
      // (2d+1)^2 <= 8y+1 < (2d+3)^2 and d = (isqrt(8y+1) - 1) / 2 exactly;
      // the lower triangle is the upper one turned by 180 degrees.  (Every
      // intermediate is non-negative, so 32-bit index code can evaluate it.)
      i64 nn = n[0];
      i64 S = nn * (nn + 1) / 2;
      V upper = al.lt(x, al.c(S));
      V y = al.sel(upper, x, al.sub(al.c(nn * nn - 1), x));
      V d = al.div(al.sub(al.isqrt(al.add(al.mulc(y, 8), al.c(1))), al.c(1)), 2);
      V i = al.sub(y, al.div(al.mul(d, al.add(d, al.c(1))), 2));
      V j = al.sub(d, i);
      return {al.sel(upper, i, al.sub(al.c(nn - 1), i)), al.sel(upper, j, al.sub(al.c(nn - 1), j))};
    }
  }
  throw std::logic_error("unknown GenP");
}

}  // namespace lego
