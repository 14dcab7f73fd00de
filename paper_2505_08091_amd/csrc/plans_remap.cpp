// Planning of index-map evaluation and layout remap kernels.
#include <algorithm>
#include <functional>
#include <map>
#include <numeric>
#include <set>
#include <sstream>
#include <stdexcept>

#include "errors.hpp"
#include "lower.hpp"
#include "plans.hpp"
#include "tune.hpp"

namespace lego {

namespace {

const char* elem_type(int bytes) {
  switch (bytes) {
    case 1: return "unsigned char";
    case 2: return "unsigned short";
    case 4: return "unsigned int";
    case 8: return "unsigned long long";
  }
  throw std::invalid_argument("element size must be 1, 2, 4 or 8 bytes");
}

std::string header() { return std::string(prelude_text()); }

// Emit every function with one common index type (64-bit if any needs it).
// Functions named in `parts` are parts of one additive split and all come from
// the expanded lowering (the form the split was proven on).
std::string emit_all(std::vector<std::pair<std::string, std::function<FnSpec(Ctx&)>>> fns, bool* wide_out,
                     std::string* info, const std::vector<std::string>& parts = {}) {
  auto variant = [&](const std::string& n) { return std::find(parts.begin(), parts.end(), n) != parts.end() ? 0 : -1; };
  bool wide = false;
  for (auto& f : fns) wide = wide || emit_best(f.first, f.second, false, variant(f.first)).wide;
  std::string code;
  for (auto& f : fns) {
    Emitted e = emit_best(f.first, f.second, wide, variant(f.first));
    code += e.code;
    if (info) *info += " " + f.first + ":" + std::to_string(e.ops) + "ops";
  }
  *wide_out = wide;
  return code;
}

}  // namespace

KernelPlan plan_index_eval(const Layout& l, int which, int idx_bytes) {
  if (idx_bytes != 4 && idx_bytes != 8) throw std::invalid_argument("idx_bytes must be 4 or 8");
  KernelPlan k;
  bool wide = false;
  std::string info;
  std::string fns;
  long long n = which == 0 ? l.size() : l.phys_size();
  if (idx_bytes == 4 && std::max(l.size(), l.phys_size()) > (1ll << 31))
    throw std::invalid_argument("int32 output cannot hold this layout's indices");
  if (which == 0) {
    fns = emit_all({{"lego_map", [&](Ctx& c) { return spec_apply_flat(c, l); }}}, &wide, &info);
  } else {
    fns = emit_all({{"lego_inv",
                     [&](Ctx& c) {
                       FnSpec f = spec_inv_flat(c, l);
                       f.out_array = true;
                       return f;
                     }}},
                   &wide, &info);
  }
  // Ordinary stores and one vector per thread (a grid covering every output
  // vector, the loop only for grids beyond 2^24 workgroups): 6.7 TB/s on the
  // 8192^2 maps, the speed of a plain fill, against 5.2 TB/s with streaming
  // stores from a 16384-workgroup grid-stride loop.
  int nt_store = 0;
  nt_store = tune("index.nt_store", nt_store) != 0;
  long long max_grid = 1ll << 24;
  max_grid = std::max(1ll, (long long)tune("index.grid", max_grid));
  std::ostringstream s;
  s << header() << "#define NT_STORE " << nt_store << "\n#define IDX_T " << (wide ? "i64" : "u32") << "\n#define OUT_T "
    << (idx_bytes == 4 ? "int" : "long long") << "\n#define PPT " << 16 / idx_bytes << "\n#define RANK "
    << l.dims().size() << "\n#define NPOINTS "
    << n << "ull\n#define " << (which == 0 ? "LEGO_HAVE_APPLY" : "LEGO_HAVE_INV") << " 1\n"
    << fns << "// ---- template ----\n" << tpl_index_eval;
  k.src = s.str();
  k.kernel = which == 0 ? "lego_apply_all" : "lego_inv_all";
  k.block = 256;
  // outputs per workgroup per round: 256 threads x one 16-byte vector
  const long long per_block = 256ll * (16 / idx_bytes);
  const long long nout = which == 0 ? n : n * (long long)l.dims().size();
  k.grid = std::max(1ll, std::min((nout + per_block - 1) / per_block, max_grid));
  k.info = std::string(which == 0 ? "apply" : "inv") + (wide ? " i64" : " u32") + info;
  return k;
}

namespace {

struct Dg {
  i64 a, b, c;  // destination weight, size, source weight
  bool tile = false;
};

// Split digit k at factor f: (a, f, c) and (a*f, b/f, c*f).
void split_digit(std::vector<Dg>& d, size_t k, i64 f) {
  Dg lo = d[k], hi = d[k];
  lo.b = f;
  hi.a = d[k].a * f;
  hi.b = d[k].b / f;
  hi.c = d[k].c * f;
  d[k] = lo;
  d.insert(d.begin() + k + 1, hi);
}

// The factor of b to take into a tile that may grow by at most `room`: the
// divisor f <= room of b with the most factors of two (so vector runs stay
// powers of two), the largest such; 1 if none.
i64 tile_factor(i64 b, i64 room) {
  i64 best = 1;
  auto twos = [](i64 x) {
    int t = 0;
    while (x % 2 == 0) x /= 2, ++t;
    return t;
  };
  for (i64 f = 2; f <= std::min(b, room); ++f)
    if (b % f == 0 && (twos(f) > twos(best) || (twos(f) == twos(best) && f > best))) best = f;
  return best;
}

// Mark the lowest digits (by destination weight if by_dst, else by source
// weight) while their product stays within `target`, splitting the first
// digit that does not fit at a factor that does.  The product never exceeds
// `target` (with extents that have no small factors it may stay below it).
void take_lowest(std::vector<Dg>& d, i64 target, bool by_dst) {
  for (;;) {
    std::vector<size_t> order(d.size());
    for (size_t k = 0; k < d.size(); ++k) order[k] = k;
    std::sort(order.begin(), order.end(), [&](size_t x, size_t y) { return by_dst ? d[x].a < d[y].a : d[x].c < d[y].c; });
    i64 cum = 1;
    bool again = false;
    for (size_t k : order) {
      if (cum >= target) break;
      if (d[k].tile) {  // taken already (by the other side's selection)
        if (cum * d[k].b > target) break;
        cum *= d[k].b;
        continue;
      }
      if (cum * d[k].b <= target) {
        d[k].tile = true;
        cum *= d[k].b;
        continue;
      }
      const i64 f = tile_factor(d[k].b, target / cum);
      if (f > 1) {
        split_digit(d, k, f);
        again = true;  // indices changed; re-run the selection
      }
      break;
    }
    if (!again) return;
  }
}

i64 tile_size(const std::vector<Dg>& d) {
  i64 t = 1;
  for (auto& x : d)
    if (x.tile) t *= x.b;
  return t;
}

int pow2_vec(i64 run, int max_elems) {
  int v = 1;
  while (v * 2 <= max_elems && run % (v * 2) == 0) v *= 2;
  return v;
}

}  // namespace

static RemapPlan plan_remap_impl(const Layout& src, const Layout& dst, int elem_bytes, bool allow_lds);

RemapPlan plan_remap(const Layout& src, const Layout& dst, int elem_bytes) {
  try {
    return plan_remap_impl(src, dst, elem_bytes, true);
  } catch (const Unsupported&) {
    // No LDS tiling fits this digit structure: fall back to the direct/gather kernel.
    return plan_remap_impl(src, dst, elem_bytes, false);
  }
}

// Box-staged remap for 2-D maps without digit structure (an element gather
// otherwise; e.g. Row <-> antidiagonal order).  A 64 x 64 box of the logical
// index space goes through LDS.  Each side is copied line by line, a line
// being a row, a column or an antidiagonal of the box with a wave's lanes
// along it; for each side the planner picks the kind of line under which that
// side's layout is most contiguous (counting, on the host, the breaks in the
// address sequence of a sample box).  It then tries to split the side's
// element offset L(64 bi + a, 64 bj + b) into a part of (box, line) and a part
// of the lane, so that an element costs one add: along an antidiagonal a + b
// is the line's, and the antidiagonal order of Figure 7 is then the line's
// start plus the row.  Returns false when no kind of line gives runs of 8
// elements on average on both sides.
static bool plan_remap_box(const Layout& src, const Layout& dst, int elem_bytes, RemapPlan* out) {
  const std::vector<i64> n = src.dims();
  if (n.size() != 2) return false;
  if (n[0] < 64 || n[1] < 64) return false;
  // Remaps whose traffic exceeds the 256 MB last-level cache go to HBM: there
  // 128 x 128 boxes (longer runs per row visited, fewer partly written cache
  // lines along antidiagonals); smaller remaps keep 64 x 64 boxes (more of
  // them in flight: 4096^2 fp32 antidiagonal -> Row 5.3 -> 6.1 TB/s), as do
  // 8-byte elements (LDS and registers).
  const bool beyond_llc = 2 * n[0] * n[1] * elem_bytes > (i64(256) << 20);
  const i64 B = tune("remap.box_side", beyond_llc && n[0] >= 128 && n[1] >= 128 && elem_bytes <= 4 ? 128 : 64);
  const char* names[3] = {"rows", "cols", "antidiags"};
  // Box element (a, b) of lane l on line p: row p, column p, or the pair of
  // antidiagonals p and p + 64 (a + b = p for l <= p, p + 64 after), whose
  // lengths add up to 64.  r: the row, column or antidiagonal it lies on.
  auto pt = [&](int ord, i64 p, i64 l, i64* a, i64* b) {
    if (ord == 0) *a = p, *b = l;
    else if (ord == 1) *a = l, *b = p;
    else *a = l, *b = (p - l) & (B - 1);
  };
  const i64 nparts[3] = {B, B, 2 * B - 1};  // rows, columns, antidiagonals
  // A box away from the edges when there is one (the first otherwise).
  const i64 o0 = n[0] >= 3 * B ? B : 0, o1 = n[1] >= 3 * B ? B : 0;
  auto breaks = [&](const Layout& L, int ord) {
    i64 nb = 0;
    for (i64 p = 0; p < B; ++p) {
      i64 prev = 0;
      for (i64 l = 0; l < B; ++l) {
        i64 a, b;
        pt(ord, p, l, &a, &b);
        const i64 x = host_apply(L, {o0 + a, o1 + b});
        if (l == 0 || x != prev + 1) ++nb;
        prev = x;
      }
    }
    return nb;
  };
  int os = 0, od = 0;
  i64 bs = -1, bd = -1;
  for (int k = 0; k < 3; ++k) {
    const i64 x = breaks(src, k), y = breaks(dst, k);
    if (bs < 0 || x < bs) bs = x, os = k;
    if (bd < 0 || y < bd) bd = y, od = k;
  }
  if (bs * 8 > B * B || bd * 8 > B * B) return false;
  // LDS slot of box element (a, b): a * (B + pad) + b, with the pad that
  // keeps the lanes of a wave on distinct 4-byte banks under both kinds of
  // line where it can (rows: stride 1; columns: B + pad; antidiagonals:
  // B + pad - 1).
  int pad = 0;
  {
    int best = 1 << 30;
    for (int pd = 0; pd < 4; ++pd) {
      int cost = 0;
      for (int k : {os, od})
        for (i64 p : {i64(0), B / 2}) {
          std::vector<int> hits(64, 0);
          int worst = 0;
          for (i64 l = 0; l < 64; ++l) {
            i64 a, b;
            pt(k, p, l, &a, &b);
            const i64 slot = a * (B + pd) + b;
            worst = std::max(worst, ++hits[(slot * elem_bytes / 4) % 64]);
          }
          cost += worst;
        }
      if (cost < best) best = cost, pad = pd;
    }
  }
  const int NT = 256;
  const i64 nbr = (n[0] + B - 1) / B, nbc = (n[1] + B - 1) / B, nb = nbr * nbc;
  // Box order, a layout over the grid of boxes.  A run along an antidiagonal
  // ends mid-line at a box edge and the rest of the line belongs to the
  // neighbouring box (above, below, left or right) along that antidiagonal:
  // the two write or fetch the shared line once each unless it meets both in
  // one L2 while it is still there.  Workgroups are dispatched round-robin
  // over the 8 XCDs, and XCD x takes the x-th eighth of the order; with the
  // grid in 2 x 2 tiles of (n/2) x (n/2) boxes, each eighth is a compact
  // (n/4) x (n/2) rectangle of boxes, walked row by row.  When an XCD holds
  // too few boxes at once for a box and the one below it to run together
  // (fewer than 8 rows of the rectangle: 128 x 128 fp32 boxes, two per CU),
  // a destination in antidiagonal order walks the rectangle in bands of 4
  // rows, column by column, so that neighbours run close in time and the
  // partial lines merge in the L2 (8192^2 fp32 forward: writes +13.5% ->
  // +4.4% over the algorithmic bytes, 5.40-5.45 -> 5.52-5.54 TB/s; reading
  // antidiagonals, the row-by-row walk measured faster).  Measured against
  // the antidiagonal order of the boxes (8192^2 fp32: 5.32 / 6.02 -> 5.52 /
  // 6.66 TB/s; 4096^2: 5.33 / 5.99 -> 5.72 / 5.95), Morton order and tiles
  // of 8 or 16 boxes.
  const bool ad_lines = os == 2 || od == 2;
  const bool xcd = nb % 8 == 0;
  long long bt = ad_lines && nbr == nbc && nbr % 2 == 0 && xcd ? nbr / 2 : 0;
  bt = tune("remap.box_tile", bt);
  const bool ad_boxes = bt > 0 && nbr % bt == 0 && nbc % bt == 0;
  const i64 per_cu = std::max<i64>(1, std::min<i64>(8, (160 * 1024) / (B * B * elem_bytes)));
  long long band = od == 2 && 32 * per_cu < 8 * bt ? 4 : 0;
  band = tune("remap.box_band", band);
  LayoutP Wb = ad_boxes ? make_tileorderby({make_row({nbr / bt, nbc / bt}), make_row({bt, bt})})
                        : make_from_piece(make_row({nbr, nbc}));
  if (ad_boxes && band > 0 && bt % band == 0)
    Wb = make_tileorderby({make_row({nbr / bt, nbc / bt}), make_row({bt / band, 1}), make_col({band, bt})});
  else
    band = 0;
  auto box_fn = [&](Ctx& c) {
    int b = c.var("b", nb);
    SymAlg al{&c};
    Sum pos = var(c, b);
    if (xcd) pos = add(c, mulc(c, fmod(c, var(c, b), 8), nb / 8), fdiv(c, var(c, b), 8));
    FnSpec f;
    f.params = {b};
    f.outs = Wb->inv(al, pos);
    f.out_bound = {nbr, nbc};
    return f;
  };
  // Element offset of lane l on row, column or antidiagonal r of box (bi,
  // bj) as a Sum (on antidiagonal r the lane's element is (l, r - l)), and its
  // split into a (box, r) part and a lane part.
  auto side = [&](Ctx& c, const Layout& L, int ord, int* bi, int* bj, int* r, int* l) {
    *bi = c.var("bi", nbr);
    *bj = c.var("bj", nbc);
    *r = c.var("r", nparts[ord]);
    *l = c.var("l", B);
    Sum a, b;
    if (ord == 0) a = var(c, *r), b = var(c, *l);
    else if (ord == 1) a = var(c, *l), b = var(c, *r);
    else a = var(c, *l), b = sub(c, var(c, *r), var(c, *l));
    SymAlg al{&c};
    return L.apply(al, {add(c, mulc(c, var(c, *bi), B), a), add(c, mulc(c, var(c, *bj), B), b)});
  };
  auto separable = [&](const Layout& L, int ord) {
    try {
      Ctx c;
      int bi, bj, r, l;
      Sum off = side(c, L, ord, &bi, &bj, &r, &l), lane, rest;
      return split_by(off, {l}, &lane, &rest);
    } catch (const std::exception&) {
      return false;
    }
  };
  const bool ssep = separable(src, os), dsep = separable(dst, od);
  auto part_fn = [&](const Layout* L, int ord, bool lane_part) {
    return [&, L, ord, lane_part](Ctx& c) {
      int bi, bj, r, l;
      Sum off = side(c, *L, ord, &bi, &bj, &r, &l), lane, rest;
      FnSpec f;
      f.valid = split_by(off, {l}, &lane, &rest);
      // the kernel adds the two parts in the index type, and their total is
      // an offset of the side's buffer
      f.ring_out = L->phys_size() <= (i64(1) << 32);
      if (lane_part) {
        f.params = {l};
        f.outs = {lane};
      } else {
        f.params = {bi, bj, r};
        f.outs = {rest};
      }
      return f;
    };
  };
  auto addr_fn = [&](const Layout* L) {
    return [&, L](Ctx& c) {
      int i = c.var("i", n[0]), j = c.var("j", n[1]);
      SymAlg al{&c};
      FnSpec f;
      f.params = {i, j};
      f.outs = {L->apply(al, {var(c, i), var(c, j)})};
      f.out_bound = {L->phys_size()};
      return f;
    };
  };
  std::vector<std::pair<std::string, std::function<FnSpec(Ctx&)>>> fns = {{"bord", box_fn}};
  std::vector<std::string> parts;
  if (ssep) {
    fns.push_back({"s_u", part_fn(&src, os, false)});
    fns.push_back({"s_l", part_fn(&src, os, true)});
    parts.insert(parts.end(), {"s_u", "s_l"});
  } else {
    fns.push_back({"s_f", addr_fn(&src)});
  }
  if (dsep) {
    fns.push_back({"d_u", part_fn(&dst, od, false)});
    fns.push_back({"d_l", part_fn(&dst, od, true)});
    parts.insert(parts.end(), {"d_u", "d_l"});
  } else {
    fns.push_back({"d_f", addr_fn(&dst)});
  }
  std::string info;
  bool wide = false;
  std::string code = emit_all(fns, &wide, &info, parts);
  // Beyond the last-level cache, the side copied along rows or columns
  // streams (non-temporal), which leaves the cache to the other side's
  // antidiagonal segments, whose partly covered lines the neighbouring boxes
  // complete (8192^2 fp32 with 128 x 128 boxes: Row <-> antidiagonal 3.9 /
  // 4.1 -> 5.3 / 5.9 TB/s; within the cache it costs 10-15%).
  int nontemporal = 0;
  if (beyond_llc && (os == 2) != (od == 2)) nontemporal = os == 2 ? 2 : 1;
  nontemporal = (int)tune("remap.nontemporal", nontemporal);
  std::ostringstream s;
  s << header() << "#define ELEM_T " << elem_type(elem_bytes) << "\n#define IDX_T " << (wide ? "i64" : "u32")
    << "\n#define BX " << B << "\n#define BPAD " << pad << "\n#define NBR " << nbr << "\n#define NBC " << nbc << "\n#define EXT0 " << n[0]
    << "\n#define EXT1 " << n[1] << "\n#define NT " << NT << "\n#define S_ORD " << os << "\n#define D_ORD " << od
    << "\n#define S_SEP " << (ssep ? 1 : 0) << "\n#define D_SEP " << (dsep ? 1 : 0) << "\n#define NONTEMPORAL "
    << nontemporal << "\n#define LEGO_REMAP_BOX 1\n"
    << code << "// ---- template ----\n" << tpl_remap;
  RemapPlan& R = *out;
  R.path = REMAP_BOX;
  R.run = 1;
  R.vec = R.vec_dst = 1;
  R.tile = B * B;
  R.kernel = "lego_remap_box";
  R.block = NT;
  R.grid = nb;
  R.src = s.str();
  R.info = "box " + std::to_string(B) + "x" + std::to_string(B) +
           (ad_boxes ? " tiles" + std::to_string(bt) + (band ? "-bands" + std::to_string(band) : "") : " row") +
           (xcd ? "-xcd" : "") + " load " + names[os] + (ssep ? " sep" : " full") + " (" + std::to_string(bs) +
           " runs) store " + names[od] + (dsep ? " sep" : " full") + " (" + std::to_string(bd) + " runs) pad " +
           std::to_string(pad) + (nontemporal & 1 ? " nt-loads" : "") + (nontemporal & 2 ? " nt-stores" : "") +
           " NT=" + std::to_string(NT) + info;
  return true;
}

static RemapPlan plan_remap_impl(const Layout& src, const Layout& dst, int elem_bytes, bool allow_lds) {
  const char* et = elem_type(elem_bytes);
  if (src.dims() != dst.dims()) throw std::length_error("remap layouts have different logical shapes");
  // Destination positions are enumerated (an ExpandBy destination has its
  // original extents only); an ExpandBy source leaves some of them without a
  // source element (Figure 9's -1): those receive zero.
  const bool masked = (bool)src.expand_inner;
  const i64 N = dst.phys_size();
  const i64 NS = src.phys_size();
  const int maxv = std::max(1, 16 / elem_bytes);
  RemapPlan R;

  // M(p) = L_src.apply(L_dst.inv(p)) in the canonical digit form.
  Ctx c0;
  int p = c0.var("p", N);
  Sum VALID;
  Sum M = remap_map_masked(c0, src, dst, p, &VALID);
  std::vector<Digit> digits;
  bool pure = !masked && N == NS && digits_of(c0, M, p, &digits);

  i64 run = 1;
  if (pure) {
    for (auto& d : digits)
      if (d.a == 1 && d.coeff == 1) run = d.b;
  }

  // Direct-path vector width: the largest V with M(V t + e) = M(V t) + e and
  // M(V t) a multiple of V, proven on the expressions (works for any layout).
  int V = 1;
  for (int v = maxv; v >= 2; v /= 2) {
    if (N % v) continue;
    Ctx c;
    int t = c.var("t", N / v), e = c.var("e", v);
    Sum pe = add(c, mulc(c, var(c, t), v), var(c, e));
    int pv = c.var("p", N);
    Sum vv;
    Sum m = subst(c, remap_map_masked(c, src, dst, pv, &vv), pv, pe);
    // A vector is either wholly inside the source's extents or wholly outside.
    if (depends_on(subst(c, vv, pv, pe), e)) continue;
    Sum ep, tp;
    if (!split_by(m, {e}, &ep, &tp)) continue;
    if (key(ep) != key(var(c, e))) continue;
    if (known_multiple(tp) % v == 0) {
      V = v;
      break;
    }
  }
  if (!pure) run = V;
  R.run = run;

  const bool long_run = run * elem_bytes >= 128 || run == N;
  if (V * elem_bytes >= 16 && (long_run || !pure)) {
    // ---- direct path
    R.path = REMAP_DIRECT;
  } else if (pure && N >= 64 && allow_lds) {
    R.path = REMAP_LDS;
  } else {
    R.path = V > 1 ? REMAP_DIRECT : REMAP_GATHER;
  }

  if (R.path == REMAP_GATHER && !masked && !dst.expand_inner && N == NS) {
    RemapPlan box;
    bool use = plan_remap_box(src, dst, elem_bytes, &box);
    use = use && tune("remap.box", 1) != 0;
    if (use) return box;
  }

  std::ostringstream s;
  std::string info;
  bool wide = false;
  // Streaming (non-temporal) loads, ordinary stores.  On MI355X this measured
  // fastest for HBM-resident tensors that are not reused by the same kernel,
  // both with caches cleaned between launches and when a remap consumes the
  // previous remap's output; cached stores leave that output in the last-level
  // cache for its consumer.  An element gather reads each source line many
  // times over neighbouring chunks, so its loads stay cached (Row <->
  // antidiagonal 4096^2 fp32: 0.74/0.97 -> 1.11/1.78 TB/s).  An LDS-staged
  // remap of at most 32 MiB per buffer streams its stores too: written
  // through the L2 of each XCD, the output of a launch this small slowed
  // the next launch that read it (2048^2 fp32 transposes alternating: 2.76 /
  // 4.42 -> 4.02 / 3.94 TB/s; Row <-> Morton 4096^2 fp16 after a cache
  // flush 4.43 / 4.73 -> 4.92 / 4.90, hot unchanged overall).
  int nontemporal = R.path == REMAP_GATHER ? 0 : 1;
  if (R.path == REMAP_LDS && N * elem_bytes <= (i64(32) << 20)) nontemporal = 3;
  nontemporal = (int)tune("remap.nontemporal", nontemporal);
  if (R.path == REMAP_DIRECT || R.path == REMAP_GATHER) {
    // 8 vectors in flight per thread (a 32 KiB chunk per workgroup at 16-byte
    // vectors): measured ahead of 2, 4 and 16, and of 128/512/1024 threads.
    int NT = 256, UNROLL = 8;
    NT = (int)tune("remap.nt", NT);
    const bool unroll_set = tune("remap.unroll", 0) != 0;
    UNROLL = (int)tune("remap.unroll", UNROLL);
    const i64 nvec = N / V;
    // Source vector of destination vector t, as an expression of t.
    auto src_vec_of = [&](Ctx& c, const Sum& t) {
      int pv = c.var("p", N);
      Sum vv;
      return fdiv(c, subst(c, remap_map_masked(c, src, dst, pv, &vv), pv, mulc(c, t, V)), V);
    };
    // A map that is not a digit permutation (a GenP, ExpandBy, ...) can cost
    // far more than a vector copy per vector.  When the map splits additively
    // into a chunk part and an in-chunk part, the chunk part is computed once
    // per workgroup: take the largest chunk (8, 4, 2 or 1 vectors per thread)
    // for which it does.
    bool src_sep = false;
    if (!pure) {
      for (int u : {8, 4, 2, 1}) {
        if (unroll_set && u != UNROLL) continue;
        const i64 ch = (i64)NT * u;
        if (nvec % ch) continue;
        Ctx c;
        int cb = c.var("c", nvec / ch), r = c.var("r", ch);
        Sum F, G;
        if (split_by(src_vec_of(c, add(c, mulc(c, var(c, cb), ch), var(c, r))), {cb}, &F, &G)) {
          UNROLL = u;
          src_sep = true;
          break;
        }
      }
    }
    const i64 chunk = (i64)NT * UNROLL;
    const i64 nblk = (nvec + chunk - 1) / chunk;
    // Chunk order.  For a digit map whose chunks are whole digits, the
    // workgroups enumerate the chunk digits by source weight (source order);
    // otherwise they run in destination order.
    std::vector<Dg> cd;  // digits of the chunk index: (dst weight in chunks, size, src weight)
    bool src_order = pure && nvec % chunk == 0;
    src_order = src_order && tune("remap.order", 1) != 0;
    if (src_order) {
      std::vector<Dg> d;
      for (auto& x : digits) d.push_back({x.a, x.b, x.coeff});
      std::sort(d.begin(), d.end(), [](const Dg& x, const Dg& y) { return x.a < y.a; });
      const i64 cel = chunk * V;  // elements per chunk
      for (size_t k = 0; k < d.size() && src_order; ++k) {
        if (d[k].a >= cel) {
          if (d[k].a % cel) src_order = false;
          cd.push_back({d[k].a / cel, d[k].b, d[k].c});
        } else if (d[k].a * d[k].b > cel) {
          i64 f = cel / d[k].a;
          if (cel % d[k].a || d[k].b % f) {
            src_order = false;
          } else {
            cd.push_back({1, d[k].b / f, d[k].c * f});
          }
        }
      }
      std::sort(cd.begin(), cd.end(), [](const Dg& x, const Dg& y) { return x.c < y.c; });
    }
    // In destination order, workgroups are dispatched round-robin over the 8
    // XCDs (each with its own L2): an element gather gives XCD x the x-th
    // eighth of the chunks, so neighbouring chunks, which such a map reads
    // from neighbouring source lines, share one L2.
    // (Measured on the element-gather path: Row <-> antidiagonal 4096^2 fp32
    // 0.42/0.63 -> 0.74/0.98 TB/s; vector maps gain nothing from it.)
    bool xcd_blocks = !src_order && !pure && nblk % 8 == 0 && R.path == REMAP_GATHER;
    xcd_blocks = xcd_blocks && tune("remap.xcd", 1) != 0;
    std::vector<std::pair<std::string, std::function<FnSpec(Ctx&)>>> dfns = {{"blk",
                                 [&](Ctx& c) {
                                   int b = c.var("b", nblk);
                                   Sum o = var(c, b);
                                   if (xcd_blocks)
                                     o = add(c, mulc(c, fmod(c, var(c, b), 8), nblk / 8), fdiv(c, var(c, b), 8));
                                   if (src_order) {
                                     o = cst(0);
                                     i64 w = 1;
                                     for (auto& x : cd) {
                                       o = add(c, o, mulc(c, fmod(c, fdiv(c, var(c, b), w), x.b), x.a));
                                       w *= x.b;
                                     }
                                   }
                                   FnSpec f;
                                   f.params = {b};
                                   f.outs = {o};
                                   return f;
                                 }},
                                {"src_vec",
                                 [&](Ctx& c) {
                                   int t = c.var("t", nvec);
                                   int pv = c.var("p", N);
                                   Sum vv;
                                   Sum m = subst(c, remap_map_masked(c, src, dst, pv, &vv), pv, mulc(c, var(c, t), V));
                                   FnSpec f;
                                   f.params = {t};
                                   f.outs = {fdiv(c, m, V)};
                                   return f;
                                 }}};
    // (declared at this scope: the builders run later, inside emit_all)
    auto part = [&](Ctx& c, bool base) {
      int cb = c.var("c", nblk), r = c.var("r", chunk);
      Sum F, G;
      FnSpec f;
      f.valid = split_by(src_vec_of(c, add(c, mulc(c, var(c, cb), chunk), var(c, r))), {cb}, &F, &G);
      f.params = {base ? cb : r};
      f.outs = {base ? F : G};
      return f;
    };
    if (src_sep) {
      dfns.push_back({"src_base", [&](Ctx& c) { return part(c, true); }});
      dfns.push_back({"src_loc", [&](Ctx& c) { return part(c, false); }});
    }
    if (masked)
      dfns.push_back({"src_ok", [&](Ctx& c) {
                        int t = c.var("t", nvec);
                        int pv = c.var("p", N);
                        Sum vv;
                        remap_map_masked(c, src, dst, pv, &vv);
                        FnSpec f;
                        f.params = {t};
                        f.outs = {subst(c, vv, pv, mulc(c, var(c, t), V))};
                        return f;
                      }});
    std::string fns = emit_all(dfns, &wide, &info, {"src_base", "src_loc"});
    s << header() << "#define ELEM_T " << et << "\n#define IDX_T " << (wide ? "i64" : "u32") << "\n#define V " << V
      << "\n#define SRC_SEP " << (src_sep ? 1 : 0)
      << "\n#define NVEC " << nvec << "ull\n#define NBLK " << nblk << "ull\n#define NT " << NT << "\n#define UNROLL " << UNROLL
      << "\n#define NONTEMPORAL " << nontemporal << "\n#define MASKED " << (masked ? 1 : 0) << "\n#define NSRC " << NS
      << "ull\n#define LEGO_REMAP_DIRECT 1\n"
      << fns << "// ---- template ----\n" << tpl_remap;
    R.kernel = "lego_remap_direct";
    R.block = NT;
    // Optionally a persistent grid: `persist` workgroups per CU loop over the chunks.
    int persist = 0;
    persist = (int)tune("remap.persist", persist);
    R.grid = persist > 0 ? std::min<i64>(nblk, 256ll * persist) : nblk;
    R.vec = V;
    R.vec_dst = V;
    R.src = s.str();
    R.info = std::string(R.path == REMAP_DIRECT ? "direct" : "gather") +
             (src_order ? " src-order" : (xcd_blocks ? " dst-order-xcd" : " dst-order")) +
             " NT=" + std::to_string(NT) + " UNROLL=" + std::to_string(UNROLL) + " V=" + std::to_string(V) +
             (src_sep ? " chunk-base" : "") +
             " run=" + std::to_string(run) + (masked ? " masked" : "") + info;
    return R;
  }

  // ---- LDS path: choose the tile digits.
  std::vector<Dg> d;
  for (auto& x : digits) d.push_back({x.a, x.b, x.coeff});
  // A remap whose traffic exceeds the 256 MB last-level cache streams from HBM:
  // there tiles taken in source order measured fastest, 32 KiB in general
  // (3-D bricks, Morton) and 64 KiB when the map keeps no two neighbours
  // together (run 1, a transpose: 512-byte runs on both sides of a 128x128
  // fp32 tile, +9-13% over 32 KiB on the 8192^2 fp32 transpose); smaller
  // remaps keep 16 KiB tiles in destination order.
  // A map that keeps no two neighbours together (run 1) takes the large
  // source-order tiles also below that size once they still give every CU
  // four tiles (4096^2 fp32 transpose: 4.89/5.34 -> 5.32/6.11 TB/s; at 2048^2,
  // 256 such tiles, the 16 KiB tiles stay ahead).
  const bool hbm_bound =
      2 * N * elem_bytes > (256ll << 20) || (run == 1 && N * elem_bytes >= 1024ll * 64 * 1024);
  i64 tile_bytes = hbm_bound ? (run == 1 ? 64 * 1024 : 32 * 1024) : 16 * 1024;
  tile_bytes = std::max<i64>(256, tune("remap.tile_bytes", tile_bytes));
  const i64 max_tile = std::min<i64>(N, std::max<i64>(32 * 1024, tile_bytes) / elem_bytes);
  i64 tdst = std::min<i64>(N, std::max<i64>(maxv, 256 / elem_bytes));
  i64 tsrc = std::min<i64>(N, std::max<i64>(maxv, 256 / elem_bytes));
  take_lowest(d, tdst, true);
  take_lowest(d, tsrc, false);
  // Grow the tile toward 16 KiB by alternately extending both sides.
  for (int step = 0; step < 16 && tile_size(d) * elem_bytes < tile_bytes; ++step) {
    std::vector<Dg> trial = d;
    if (step % 2 == 0)
      tdst *= 2;
    else
      tsrc *= 2;
    take_lowest(trial, step % 2 == 0 ? tdst : tsrc, step % 2 == 0);
    if (tile_size(trial) > max_tile) break;
    d = trial;
  }
  std::sort(d.begin(), d.end(), [](const Dg& x, const Dg& y) { return x.a < y.a; });
  const i64 TILE = tile_size(d);
  // never emit a tile beyond 128 KiB of LDS (160 KiB per CU)
  if (TILE * elem_bytes > (128 << 10)) throw Unsupported("remap LDS tile exceeds 128 KiB");
  const i64 G = N / TILE;
  // Tile-local orders and weights (recomputed after the digit splits below).
  std::vector<size_t> td, ts, gd;
  std::vector<i64> wd, ws, wg;
  bool lds_src_order = hbm_bound;
  lds_src_order = tune("remap.order", lds_src_order) != 0;
  auto orders = [&]() {
    td.clear(), ts.clear(), gd.clear();
    for (size_t k = 0; k < d.size(); ++k) (d[k].tile ? td : gd).push_back(k);
    // Tile order (the digit layout over tiles): source order for HBM-bound
    // remaps, destination order otherwise.
    if (lds_src_order) std::sort(gd.begin(), gd.end(), [&](size_t x, size_t y) { return d[x].c < d[y].c; });
    ts = td;
    std::sort(ts.begin(), ts.end(), [&](size_t x, size_t y) { return d[x].c < d[y].c; });
    wd.assign(d.size(), 0), ws.assign(d.size(), 0), wg.assign(d.size(), 0);
    i64 w = 1;
    for (size_t k : td) wd[k] = w, w *= d[k].b;
    w = 1;
    for (size_t k : ts) ws[k] = w, w *= d[k].b;
    w = 1;
    for (size_t k : gd) wg[k] = w, w *= d[k].b;
  };
  orders();
  // Vector widths: the leading tile digits that are contiguous on the source
  // (destination) side form runs; vectors must divide those runs.
  i64 srun = 1, drun = 1;
  for (size_t k : ts) {
    if (d[k].c != srun) break;
    srun *= d[k].b;
  }
  for (size_t k : td) {
    if (d[k].a != drun) break;
    drun *= d[k].b;
  }
  const int VL = pow2_vec(srun, maxv);
  const int VS = pow2_vec(drun, maxv);
  // Split tile digits so that a source vector (the lowest VL of the tile's
  // source order) and a destination vector (the lowest VS of its destination
  // order) are made of whole digits.  Splitting a digit keeps the map; it
  // only names the sub-ranges the block transfer below works with.
  bool whole = true;
  for (bool split = true; split && whole;) {
    split = false;
    for (int side = 0; side < 2 && !split && whole; ++side) {
      i64 rem = side == 0 ? VL : VS;
      for (size_t k : side == 0 ? ts : td) {
        if (rem == 1) break;
        if (rem % d[k].b == 0) {
          rem /= d[k].b;
          continue;
        }
        if (d[k].b % rem == 0) {
          split_digit(d, k, rem);
          orders();
          split = true;
        } else {
          whole = false;
        }
        break;
      }
    }
  }
  // Digit classes: in the source vector (VL), in the destination vector (VS).
  std::vector<char> in_vl(d.size()), in_vs(d.size());
  if (whole) {
    i64 r = 1;
    for (size_t k : ts)
      if (r < VL) in_vl[k] = 1, r *= d[k].b;
    r = 1;
    for (size_t k : td)
      if (r < VS) in_vs[k] = 1, r *= d[k].b;
  }
  // Block transfer: a thread loads the NX source vectors that together hold
  // NY whole destination vectors (the destination-vector digits outside the
  // source vector, X, index the loads; the source-vector digits outside the
  // destination vector, Y, index the stores), permutes them in registers,
  // and writes whole destination vectors into LDS.  Both LDS phases are then
  // vector accesses.  Taken when a destination vector spans several source
  // vectors (a transposing tile) and a block fits a thread's share.
  std::vector<size_t> xd, yd, bd;  // X (destination order), Y (source order), the rest (source order)
  for (size_t k : td)
    if (whole && in_vs[k] && !in_vl[k]) xd.push_back(k);
  for (size_t k : ts) {
    if (!whole) break;
    if (in_vl[k] && !in_vs[k]) yd.push_back(k);
    if (!in_vl[k] && !in_vs[k]) bd.push_back(k);
  }
  i64 NX = 1, NY = 1;
  for (size_t k : xd) NX *= d[k].b;
  for (size_t k : yd) NY *= d[k].b;
  const i64 BLK = VL * NX;
  // The loads stay coalesced only if the lanes of one load instruction, which
  // walk the remaining digits in source order, cover whole 128-byte lines: a
  // destination-vector digit low in the source order (Morton -> row) would
  // leave gaps between the lanes' vectors.
  i64 lane_run = VL;
  for (size_t k : bd) {
    if (d[k].c != lane_run) break;
    lane_run *= d[k].b;
  }
  bool block = whole && NX >= 2 && VS >= 2 && BLK == VS * NY && BLK <= 64 && TILE % BLK == 0 &&
               lane_run * elem_bytes >= 128;
  block = block && tune("remap.block", 1) != 0;
  std::vector<i64> wx(d.size()), wy(d.size()), wb(d.size());
  {
    i64 w = 1;
    for (size_t k : xd) wx[k] = w, w *= d[k].b;
    w = 1;
    for (size_t k : yd) wy[k] = w, w *= d[k].b;
    w = 1;
    for (size_t k : bd) wb[k] = w, w *= d[k].b;
  }
  // LDS tile rows of 256 bytes, in destination order.  The
  // destination-side VS-vectors of a row are XOR-swizzled across rows (the
  // swizzle is itself a GenP layout over [TILE/W, W]): vector v of row r goes
  // to position v ^ ((r / S) % (W / VS)).  S is chosen below by counting the
  // bank conflicts of both LDS phases of one tile.
  auto row_of = [&](i64 bytes) {
    i64 w = std::max<i64>(VS, bytes / elem_bytes);
    while (w > VS && TILE % w) w /= 2;
    return w;
  };
  auto swizzles = [&](i64 w) { return w / VS >= 2 && ((w / VS) & (w / VS - 1)) == 0 && TILE % w == 0; };
  i64 W = row_of(256);
  bool swz = swizzles(W);
  auto digit_of = [&](Ctx& c, const Sum& x, i64 weight, i64 b) { return fmod(c, fdiv(c, x, weight), b); };
  auto kd_from_ks = [&](Ctx& c, const Sum& ks) {
    Sum kd = cst(0);
    for (size_t k : ts) kd = add(c, kd, mulc(c, digit_of(c, ks, ws[k], d[k].b), wd[k]));
    return kd;
  };
  // Are the VL elements of a source vector consecutive in destination order
  // (then they stay contiguous in LDS under any vector-granular swizzle)?
  bool contig = false;
  {
    Ctx c;
    int q = c.var("q", TILE / VL), e = c.var("e", VL);
    Sum kd = kd_from_ks(c, add(c, mulc(c, var(c, q), VL), var(c, e)));
    Sum ep, qp;
    if (split_by(kd, {e}, &ep, &qp) && key(ep) == key(var(c, e))) {
      contig = known_multiple(qp) % VL == 0;
    }
  }
  // A VL-run longer than a swizzled VS-vector may be split by the swizzle.
  if (VL > VS && swz) contig = false;
  if (contig) block = false;
  // Threads per workgroup: the largest divisor of both vector (block) counts
  // up to 256 (whole passes over the tile on either side); at least one wave.
  const i64 nvg = std::gcd(TILE / (block ? BLK : VL), TILE / VS);
  int NT = 1;
  for (int t = 256; t >= 1; --t)
    if (nvg % t == 0) {
      NT = t;
      break;
    }
  if (NT < 64 && NT != nvg) throw Unsupported("LDS tile does not divide into vectors");
  // each thread holds TILE / NT elements in registers between the two phases
  if (TILE * elem_bytes / NT > 512) throw Unsupported("LDS tile too large for its thread count");
  // Bank conflicts of one tile under the swizzle strides, counted on the
  // host: a write of A bytes per lane is served 128/A lanes at a time over 32
  // banks of 4 bytes, a read 256/A lanes at a time over 64 banks (all 64
  // lanes for narrower accesses), and a group costs as many passes as the
  // most distinct dwords any one bank receives in it.  (The write rule
  // reproduces the LDS bank-conflict cycles counted on gfx950 for the
  // scattered and block writes of transposes and Morton orders, the read
  // rule the conflict-free 16-byte fragment reads of the GEMM.)
  auto dig = [&](i64 x, i64 weight, i64 b) { return (x / weight) % b; };
  auto kd_num = [&](i64 ks) {
    i64 kd = 0;
    for (size_t k : ts) kd += dig(ks, ws[k], d[k].b) * wd[k];
    return kd;
  };
  // The XOR key of LDS row r: (r / S) % K with K = W / VS (the XOR-swizzle
  // GenP over [TILE / W, W]), optionally XORed with (r / S2) % K for a second
  // stride S2 > S (0: none), which separates lanes whose rows differ in bits
  // that one window of the row index does not cover.
  i64 swz_s2 = 0;
  auto key_num = [&](i64 r, i64 S, i64 S2) {
    const i64 K = W / VS;
    return ((r / S) % K) ^ (S2 ? (r / S2) % K : 0);
  };
  auto slot_num = [&](i64 kd, i64 S, i64 S2) {
    if (!swz) return kd;
    const i64 r = kd / W, col = kd % W;
    return r * W + (((col / VS) ^ key_num(r, S, S2)) * VS) + col % VS;
  };
  auto passes = [&](const std::vector<i64>& slot, int bytes, bool read) {  // one instruction of one wave
    const int window = read ? 256 : 128;
    const int gsz = (int)std::min<i64>(64, std::max(1, window / bytes));
    i64 total = 0;
    for (size_t g0 = 0; g0 < slot.size(); g0 += gsz) {
      std::map<i64, std::set<i64>> bank;
      for (size_t l = g0; l < std::min(slot.size(), g0 + gsz); ++l)
        for (i64 dw = slot[l] * elem_bytes / 4; dw <= (slot[l] * elem_bytes + bytes - 1) / 4; ++dw)
          bank[dw % (window / 4)].insert(dw);
      size_t m = 1;
      for (auto& kv : bank) m = std::max(m, kv.second.size());
      total += (i64)m;
    }
    return total;
  };
  auto conflicts = [&](i64 S, i64 S2, i64* wr, i64* rd) {
    *wr = *rd = 0;
    std::vector<i64> sl;
    const i64 nq = block ? TILE / BLK : TILE / VL;
    for (i64 q0 = 0; q0 < nq; q0 += 64) {  // one wave's instruction
      const i64 lanes = std::min<i64>(64, nq - q0);
      const i64 ninst = block ? NY : (contig ? 1 : VL);
      for (i64 u = 0; u < ninst; ++u) {
        sl.clear();
        for (i64 l = 0; l < lanes; ++l) {
          const i64 q = q0 + l;
          i64 kd = 0;
          if (block) {
            for (size_t k : bd) kd += dig(q, wb[k], d[k].b) * wd[k];
            for (size_t k : yd) kd += dig(u, wy[k], d[k].b) * wd[k];
          } else {
            kd = kd_num(q * VL + u);
          }
          sl.push_back(slot_num(kd, S, S2));
        }
        const i64 p = passes(sl, (int)((block ? VS : contig ? VL : 1) * elem_bytes), false);
        *wr += p - (lanes + 63) / 64 * std::max<i64>(1, (block ? VS : contig ? VL : 1) * elem_bytes * 64 / 128);
      }
    }
    for (i64 q0 = 0; q0 < TILE / VS; q0 += 64) {
      sl.clear();
      for (i64 l = 0; l < std::min<i64>(64, TILE / VS - q0); ++l) sl.push_back(slot_num((q0 + l) * VS, S, S2));
      *rd += passes(sl, (int)(VS * elem_bytes), true) - std::max<i64>(1, VS * elem_bytes * 64 / 256);
    }
  };
  // Candidates: rows of 256 and of 128 bytes (the latter keep two vectors
  // half a 256-byte row apart, which share banks under any XOR of the row,
  // in different rows) and every stride S; the fewest passes win.
  i64 swz_s = contig ? 1 : VL, best_w = 0, best_r = 0;
  if (swz) {
    conflicts(swz_s, 0, &best_w, &best_r);
    const i64 W256 = W;
    // single strides first (fewer operations), pairs only if still needed
    for (int pairs = 0; pairs < 2 && best_w + best_r > 0; ++pairs)
      for (i64 wb : {256, 128}) {
        const i64 w = row_of(wb);
        if (!swizzles(w) || (wb == 128 && w == W256)) continue;
        const i64 keep = W;
        W = w;
        bool better = false;
        for (i64 S = 1; S <= TILE / W; S *= 2)
          for (i64 S2 = pairs ? 2 * S : 0; S2 <= (pairs ? TILE / W : 0); S2 = S2 ? S2 * 2 : 1) {
            i64 cw, cr;
            conflicts(S, S2, &cw, &cr);
            if (cw + cr < best_w + best_r) swz_s = S, swz_s2 = S2, best_w = cw, best_r = cr, better = true;
            if (!pairs) break;
          }
        if (!better) W = keep;
      }
  }
  swz_s = std::max<i64>(1, tune("remap.swizzle", swz_s));
  swz_s2 = std::max<i64>(0, tune("remap.swizzle2", swz_s2));
  W = row_of(tune("remap.lds_row", W * elem_bytes));
  if (swz) conflicts(swz_s, swz_s2, &best_w, &best_r);
  auto lds_slot = [&](Ctx& c, const Sum& kd) {
    if (!swz) return kd;
    const i64 K = W / VS;
    Sum r = fdiv(c, kd, W), col = fmod(c, kd, W);
    Sum key = fmod(c, fdiv(c, r, swz_s), K);
    if (swz_s2) key = bxor(c, key, fmod(c, fdiv(c, r, swz_s2), K));
    return add(c, add(c, mulc(c, r, W), mulc(c, bxor(c, fdiv(c, col, VS), key), VS)), fmod(c, col, VS));
  };
  auto group_part = [&](Ctx& c, int g, bool dst_side) {
    Sum o = cst(0);
    for (size_t k : gd) o = add(c, o, mulc(c, digit_of(c, var(c, g), wg[k], d[k].b), dst_side ? d[k].a : d[k].c));
    return o;
  };
  std::vector<std::pair<std::string, std::function<FnSpec(Ctx&)>>> fnl;
  if (block) {
    fnl.push_back({"src_off", [&](Ctx& c) {
                     int g = c.var("g", G), b = c.var("b", TILE / BLK), x = c.var("x", NX);
                     Sum o = group_part(c, g, false);
                     for (size_t k : bd) o = add(c, o, mulc(c, digit_of(c, var(c, b), wb[k], d[k].b), d[k].c));
                     for (size_t k : xd) o = add(c, o, mulc(c, digit_of(c, var(c, x), wx[k], d[k].b), d[k].c));
                     FnSpec f;
                     f.params = {g, b, x};
                     f.outs = {o};
                     return f;
                   }});
    fnl.push_back({"ldsw", [&](Ctx& c) {
                     int b = c.var("b", TILE / BLK), y = c.var("y", NY);
                     Sum kd = cst(0);
                     for (size_t k : bd) kd = add(c, kd, mulc(c, digit_of(c, var(c, b), wb[k], d[k].b), wd[k]));
                     for (size_t k : yd) kd = add(c, kd, mulc(c, digit_of(c, var(c, y), wy[k], d[k].b), wd[k]));
                     FnSpec f;
                     f.params = {b, y};
                     f.outs = {lds_slot(c, kd)};
                     return f;
                   }});
  } else {
    fnl.push_back({"src_off", [&](Ctx& c) {
                     int g = c.var("g", G), q = c.var("q", TILE / VL);
                     Sum ks = mulc(c, var(c, q), VL);
                     Sum o = group_part(c, g, false);
                     for (size_t k : ts) o = add(c, o, mulc(c, digit_of(c, ks, ws[k], d[k].b), d[k].c));
                     FnSpec f;
                     f.params = {g, q};
                     f.outs = {o};
                     return f;
                   }});
    fnl.push_back({"ldsw", [&](Ctx& c) {
                     int q = c.var("q", TILE / VL), e = c.var("e", VL);
                     Sum ks = add(c, mulc(c, var(c, q), VL), var(c, e));
                     FnSpec f;
                     f.params = {q, e};
                     f.outs = {lds_slot(c, kd_from_ks(c, ks))};
                     return f;
                   }});
  }
  fnl.push_back({"ldsr", [&](Ctx& c) {
                   int q = c.var("q", TILE / VS);
                   FnSpec f;
                   f.params = {q};
                   f.outs = {lds_slot(c, mulc(c, var(c, q), VS))};
                   return f;
                 }});
  fnl.push_back({"dst_off", [&](Ctx& c) {
                   int g = c.var("g", G), q = c.var("q", TILE / VS);
                   Sum kd = mulc(c, var(c, q), VS);
                   Sum o = group_part(c, g, true);
                   for (size_t k : td) o = add(c, o, mulc(c, digit_of(c, kd, wd[k], d[k].b), d[k].a));
                   FnSpec f;
                   f.params = {g, q};
                   f.outs = {o};
                   return f;
                 }});
  std::string fns = emit_all(fnl, &wide, &info);
  // The block's register permutation: element e of destination vector y is
  // element blk_el(y * VS + e) of the block's loads (source vector x at
  // x * VL, its element at + e).
  std::string blk_tab;
  if (block) {
    std::ostringstream t;
    t << "LEGO_FN constexpr int blk_el(int k) {\n  constexpr int t[" << NY * VS << "] = {";
    for (i64 y = 0; y < NY; ++y)
      for (i64 e = 0; e < VS; ++e) {
        // digit values of this element: Y digits from y, destination-vector digits from e
        std::vector<i64> val(d.size(), 0);
        for (size_t k : yd) val[k] = dig(y, wy[k], d[k].b);
        for (size_t k : td)
          if (in_vs[k]) val[k] = dig(e, wd[k], d[k].b);
        i64 x = 0, el = 0;
        for (size_t k : xd) x += val[k] * wx[k];
        for (size_t k : ts)
          if (in_vl[k]) el += val[k] * ws[k];
        t << (y || e ? ", " : "") << x * VL + el;
      }
    t << "};\n  return t[k];\n}\n";
    blk_tab = t.str();
  }
  s << header() << "#define ELEM_T " << et << "\n#define IDX_T " << (wide ? "i64" : "u32") << "\n#define TILE " << TILE
    << "\n#define NELEM " << N << "ull\n#define NTILES " << G << "ull\n#define NT " << NT << "\n#define VL " << VL << "\n#define VS " << VS << "\n#define LDSW_CONTIG "
    << (contig ? 1 : 0) << "\n#define LDS_BLOCK " << (block ? 1 : 0) << "\n#define NX " << NX << "\n#define NY " << NY
    << "\n#define NONTEMPORAL " << nontemporal << "\n#define LEGO_REMAP_LDS 1\n"
    << fns << blk_tab << "// ---- template ----\n" << tpl_remap;
  R.kernel = "lego_remap_lds";
  R.block = NT;
  R.grid = G;
  R.vec = VL;
  R.vec_dst = VS;
  R.tile = TILE;
  R.src = s.str();
  R.info = "lds TILE=" + std::to_string(TILE) + " VL=" + std::to_string(VL) + " VS=" + std::to_string(VS) +
           " W=" + std::to_string(W) + (swz ? " xor/" + std::to_string(swz_s) + (swz_s2 ? "^" + std::to_string(swz_s2) : "") : " row") +
           (block ? " block " + std::to_string(NX) + "x" + std::to_string(NY) : contig ? " contig" : " scatter") +
           " bank-passes+" + std::to_string(best_w) + "/" + std::to_string(best_r) +
           (lds_src_order ? " src-order" : " dst-order") +
           " run=" + std::to_string(run) + info;
  return R;
}

}  // namespace lego
