// Layout constructors and validation (Section III-B: the grammar of Figure 3,
// the correctness conditions stated after Figure 7, and the sugar after
// Equation (2)).
#include "layout.hpp"

#include "errors.hpp"

#include <algorithm>
#include <functional>
#include <sstream>

namespace lego {

IntAlg::V IntAlg::isqrt(V x) const {
  if (x <= 0) return 0;
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
  return (V)r;
}

std::vector<int> sigma_inverse(const std::vector<int>& sigma) {
  std::vector<int> inv(sigma.size());
  for (size_t k = 0; k < sigma.size(); ++k) inv[sigma[k] - 1] = (int)k + 1;
  return inv;
}

// sigma_{d x q} = flatten(A), A[k][h] = k + 1 + d*h.
std::vector<int> sigma_dq(int d, int q) {
  std::vector<int> s;
  for (int k = 0; k < d; ++k)
    for (int h = 0; h < q; ++h) s.push_back(k + 1 + d * h);
  return s;
}

i64 product(const std::vector<i64>& v) {
  i64 p = 1;
  for (i64 x : v) {
    if (x <= 0) throw std::invalid_argument("dimension sizes must be positive");
    if (p > (i64(1) << 62) / x) throw std::overflow_error("layout size overflows int64");
    p *= x;
  }
  return p;
}

int ilog2_exact(i64 x) {
  if (x <= 0 || (x & (x - 1))) return -1;
  int s = 0;
  while ((i64(1) << s) < x) ++s;
  return s;
}

static void check_dims(const std::vector<i64>& n) {
  if (n.empty()) throw std::invalid_argument("a tile needs at least one dimension");
  (void)product(n);
}

std::string Piece::describe() const {
  std::ostringstream o;
  auto vec = [&](auto& v) {
    o << "[";
    for (size_t i = 0; i < v.size(); ++i) o << (i ? "," : "") << v[i];
    o << "]";
  };
  if (regp) {
    o << "RegP(";
    vec(n);
    o << ",";
    vec(sigma);
    o << ")";
  } else {
    static const char* names[] = {"?", "morton", "xor_swizzle", "reverse", "antidiag", "expr"};
    o << "GenP(";
    vec(n);
    o << "," << names[gk];
    if (gk == GEN_EXPR) {
      o << ",\"" << ex->apply_text << "\"";
      for (auto& t : ex->inv_text) o << ",\"" << t << "\"";
    }
    if (!prm.empty()) {
      o << ",";
      vec(prm);
    }
    o << ")";
  }
  return o.str();
}

PieceP make_regp(const std::vector<i64>& n, const std::vector<int>& sigma) {
  check_dims(n);
  if (sigma.size() != n.size()) throw std::invalid_argument("sigma length differs from the tile rank");
  std::vector<int> s = sigma;
  std::sort(s.begin(), s.end());
  for (size_t k = 0; k < s.size(); ++k)
    if (s[k] != (int)k + 1) throw std::domain_error("sigma is not a permutation of [1..d]");
  auto p = std::make_shared<Piece>();
  p->regp = true;
  p->n = n;
  p->sigma = sigma;
  return p;
}

// Row([n1..nd]) = RegP(n, [1..d]).
PieceP make_row(const std::vector<i64>& n) {
  std::vector<int> s;
  for (size_t k = 0; k < n.size(); ++k) s.push_back((int)k + 1);
  return make_regp(n, s);
}

// Col([n1..nd]) = RegP([n1..nd], [d..1]): the logical dims stay [n1..nd] and
// the first index is fastest (the column-major meaning used for operands).
PieceP make_col(const std::vector<i64>& n) {
  std::vector<int> s;
  for (size_t k = n.size(); k > 0; --k) s.push_back((int)k);
  return make_regp(n, s);
}

PieceP make_genp(int kind, const std::vector<i64>& n, const std::vector<i64>& prm) {
  check_dims(n);
  auto p = std::make_shared<Piece>();
  p->regp = false;
  p->gk = kind;
  p->n = n;
  p->prm = prm;
  switch (kind) {
    case GEN_MORTON:
      if (n.size() != 2 || ilog2_exact(n[0]) < 0 || ilog2_exact(n[1]) < 0)
        throw std::invalid_argument("Morton order needs a 2D tile with power-of-two sides");
      if (!prm.empty()) throw std::invalid_argument("Morton order takes no parameters");
      break;
    case GEN_XOR_SWIZZLE: {
      if (n.size() != 2 || prm.size() != 2) throw std::invalid_argument("XOR swizzle needs [R,C] and (v, s)");
      i64 C = n[1], v = prm[0], s = prm[1];
      if (v <= 0 || s <= 0 || C % v != 0 || ilog2_exact(C / v) < 0)
        throw std::invalid_argument("XOR swizzle needs v | C, C/v a power of two and s > 0");
      break;
    }
    case GEN_REVERSE:
      if (!prm.empty()) throw std::invalid_argument("reverse takes no parameters");
      break;
    case GEN_ANTIDIAG:
      if (n.size() != 2 || n[0] != n[1]) throw std::invalid_argument("antidiagonal order needs a square 2D tile");
      if (!prm.empty()) throw std::invalid_argument("antidiagonal order takes no parameters");
      break;
    default:
      throw std::invalid_argument("unknown GenP kind");
  }
  return p;
}

PieceP make_genp_expr(const std::vector<i64>& n, const std::string& apply, const std::vector<std::string>& inv) {
  check_dims(n);
  const size_t d = n.size();
  if (inv.size() != d) throw std::invalid_argument("an expression GenP needs one inverse expression per dimension");
  std::vector<std::pair<std::string, i64>> consts;
  for (size_t k = 0; k < d; ++k) consts.push_back({"n" + std::to_string(k), n[k]});
  std::vector<std::string> fwd_vars;
  for (size_t k = 0; k < d; ++k) fwd_vars.push_back("i" + std::to_string(k));
  static const char* short_names[] = {"i", "j", "k"};
  for (size_t k = 0; k < d && k < 3; ++k) fwd_vars.push_back(short_names[k]);
  auto ex = std::make_shared<GenExpr>();
  ex->apply_text = apply;
  ex->inv_text = inv;
  // the short names alias the first coordinates: map them onto i0..i2
  GNodeP fwd = parse_gexpr(apply, fwd_vars, consts);
  std::function<GNodeP(const GNodeP&)> alias = [&](const GNodeP& g) -> GNodeP {
    auto c = std::make_shared<GNode>(*g);
    if (c->k == GNode::Var && c->var >= (int)d) c->var -= (int)d;
    for (auto& kid : c->kids) kid = alias(kid);
    return c;
  };
  ex->apply = alias(fwd);
  for (auto& t : inv) ex->inv.push_back(parse_gexpr(t, {"x"}, consts));
  auto p = std::make_shared<Piece>();
  p->regp = false;
  p->gk = GEN_EXPR;
  p->n = n;
  p->ex = ex;
  // Small tiles are checked exhaustively: f must be a bijection onto
  // [0, |tile|) and the inverse must undo it.
  const i64 N = product(n);
  if (N <= (i64(1) << 20)) {
    IntAlg al;
    std::vector<char> hit(N, 0);
    for (i64 x = 0; x < N; ++x) {
      std::vector<i64> i = unflatten(al, n, x);
      i64 f = p->apply(al, i);
      if (f < 0 || f >= N || hit[f]++) throw NotBijective("the expression GenP is not a bijection onto [0, size)");
      if (p->inv(al, f) != i) throw NotBijective("the inverse expressions do not invert the forward map");
    }
  }
  return p;
}

LayoutP make_groupby(const std::vector<i64>& dims) {
  check_dims(dims);
  auto l = std::make_shared<Layout>();
  l->g = dims;
  return l;
}

// Dot notation: base.OrderBy(pieces).  The element counts of the GroupBy and
// of every OrderBy must agree (the second correctness condition).
LayoutP make_orderby(const LayoutP& base, const std::vector<PieceP>& pieces) {
  if (!base) throw std::invalid_argument("null base layout");
  if (base->expand_inner) throw std::invalid_argument("OrderBy cannot follow ExpandBy");
  if (pieces.empty()) throw std::invalid_argument("OrderBy needs at least one permutation");
  OrderBy o;
  o.p = pieces;
  if (o.size() != base->size()) throw std::length_error("OrderBy element count differs from the GroupBy");
  auto l = std::make_shared<Layout>(*base);
  l->chain.push_back(o);
  return l;
}

// TileBy_{q x d}(T^1..T^q) = GroupBy(T^1..T^q).OrderBy(RegP(T^1..T^q, sigma_{d x q})).
LayoutP make_tileby(int q, int d, const std::vector<i64>& tiles) {
  if (q <= 0 || d <= 0 || (int)tiles.size() != q * d) throw std::invalid_argument("TileBy needs q*d tile sizes");
  return make_orderby(make_groupby(tiles), {make_regp(tiles, sigma_dq(d, q))});
}

// TileOrderBy_{q x d}(P^1..P^q) = GroupBy(N).OrderBy(RegP(I, sigma_{d x q}^{-1})).OrderBy(P^1..P^q)
// with N_k = prod_h n^h_k the full extents and I = sigma_{d x q}(tile-major
// dims) the interleaved digit dims: full coordinates go to tile-major storage
// whose level h is ordered by P^h.
LayoutP make_tileorderby(const std::vector<PieceP>& levels) {
  if (levels.empty()) throw std::invalid_argument("TileOrderBy needs at least one level");
  size_t d = levels[0]->n.size();
  for (auto& p : levels)
    if (p->n.size() != d) throw std::invalid_argument("TileOrderBy levels must have equal rank");
  int q = (int)levels.size();
  std::vector<i64> tile_major;
  for (auto& p : levels) tile_major.insert(tile_major.end(), p->n.begin(), p->n.end());
  std::vector<int> s = sigma_dq((int)d, q);
  std::vector<i64> inter = gather(s, tile_major);
  std::vector<i64> full(d, 1);
  for (auto& p : levels)
    for (size_t k = 0; k < d; ++k) full[k] *= p->n[k];
  LayoutP l = make_orderby(make_groupby(full), {make_regp(inter, sigma_inverse(s))});
  return make_orderby(l, levels);
}

LayoutP make_from_piece(const PieceP& p) { return make_orderby(make_groupby(p->n), {p}); }

LayoutP make_expandby(const std::vector<i64>& en, const std::vector<i64>& ne, const LayoutP& inner) {
  if (!inner) throw std::invalid_argument("null layout");
  if (en.size() != ne.size() || en.empty()) throw std::invalid_argument("ExpandBy extents must have equal rank");
  check_dims(en);
  if (product(ne) != inner->size()) throw std::length_error("expanded extents differ from the inner layout size");
  for (size_t k = 0; k < en.size(); ++k)
    if (en[k] > ne[k]) throw std::invalid_argument("ExpandBy must widen every extent");
  auto l = std::make_shared<Layout>();
  l->expand_inner = inner;
  l->en = en;
  l->ne = ne;
  return l;
}

i64 host_apply(const Layout& l, const std::vector<i64>& idx) {
  IntAlg al;
  return l.apply(al, idx);
}

std::vector<i64> host_inv(const Layout& l, i64 x) {
  IntAlg al;
  return l.inv(al, x);
}

}  // namespace lego
