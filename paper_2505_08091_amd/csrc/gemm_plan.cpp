// GEMM planning.  See gemm_plan.hpp and kernels/gemm.hip.
#include "gemm_plan.hpp"

#include <algorithm>
#include <cstdlib>
#include <map>
#include <mutex>
#include <sstream>
#include <tuple>

#include "errors.hpp"
#include "lower.hpp"
#include "tune.hpp"

namespace lego {

LayoutP mfma_fragment_layout(int instr, int operand) {
  if (instr == 0) {
    // v_mfma_f32_32x32x16: A/B lane l holds row (or column) l%32, k = 8*(l/32)+e;
    // C/D register r of lane l is row 8*(r/4) + 4*(l/32) + r%4, column l%32.
    if (operand == 0 || operand == 1) return make_orderby(make_groupby({64, 8}), {make_regp({2, 32, 8}, {2, 1, 3})});
    if (operand == 2) return make_orderby(make_groupby({64, 16}), {make_regp({2, 32, 4, 4}, {3, 1, 4, 2})});
  } else if (instr == 1) {
    // v_mfma_f32_16x16x32: A/B lane l holds row l%16, k = 8*(l/16)+e;
    // C/D register r of lane l is row 4*(l/16) + r, column l%16.
    if (operand == 0 || operand == 1) return make_orderby(make_groupby({64, 8}), {make_regp({4, 16, 8}, {2, 1, 3})});
    if (operand == 2) return make_orderby(make_groupby({64, 4}), {make_regp({4, 16, 4}, {1, 3, 2})});
  }
  throw std::invalid_argument("unknown MFMA instruction or operand");
}

GemmRequest gemm_request(const lego_gemm_desc& d, const std::function<LayoutP(lego_layout_t)>& resolve) {
  GemmRequest r;
  r.M = d.M;
  r.N = d.N;
  r.K = d.K;
  r.dtype = d.in_dtype;
  r.bm = d.bm;
  r.bn = d.bn;
  r.bk = d.bk;
  r.wm = d.wm;
  r.wn = d.wn;
  r.group_m = d.group_m;
  r.xcd = d.xcd_remap;
  r.stages = d.stages;
  r.a = resolve(d.a);
  r.b = resolve(d.b);
  r.c = resolve(d.c);
  r.sched = resolve(d.sched);
  r.lds_a = resolve(d.lds_a);
  r.lds_b = resolve(d.lds_b);
  r.frag_a = resolve(d.frag_a);
  r.frag_b = resolve(d.frag_b);
  r.frag_c = resolve(d.frag_c);
  return r;
}

namespace {

bool pow2(i64 x) { return x > 0 && (x & (x - 1)) == 0; }

// Two layouts with equal dims and sizes that map every logical point alike.
bool same_map(const Layout& x, const Layout& y) {
  if (x.dims() != y.dims() || x.size() != y.size()) return false;
  const std::vector<i64> n = x.dims();
  std::vector<i64> idx(n.size(), 0);
  IntAlg al;
  for (i64 f = 0; f < x.size(); ++f) {
    i64 r = f;
    for (size_t k = n.size(); k-- > 0;) {
      idx[k] = r % n[k];
      r /= n[k];
    }
    if (x.apply(al, idx) != y.apply(al, idx)) return false;
  }
  return true;
}

// Default LDS tile layout: 16-byte vectors of a row XOR-permuted by (row/s)
// mod (k/8).  A b128 fragment read is served 16 lanes (16 rows) at a time over
// 64 banks of 4 bytes, i.e. a 256-byte bank window holding 256/(2k) rows of k
// 16-bit elements; keying the XOR on row/s with s = 128/k gives the 16 rows of
// a phase distinct bank groups (s = 2 for k = 64, 4 for k = 32).
LayoutP default_lds(i64 rows, i64 k) {
  if (k % 8 == 0 && pow2(k / 8) && k / 8 >= 2) {
    i64 s = std::max<i64>(1, 128 / k);
    s = std::max<i64>(1, tune("gemm.lds_s", s));
    return make_from_piece(make_genp(GEN_XOR_SWIZZLE, {rows, k}, {8, s}));
  }
  return make_from_piece(make_row({rows, k}));
}

// LDS tile for an operand that is contiguous along m (A) or n (B) in global
// memory: stored one k-row at a time with the m/n index fastest, so global
// vectors land unchanged, and 64-byte granules of a k-row XOR-permuted by the
// k-row (a GenP over [k, rows]).  Fragments are read with the transposing LDS
// load, which fetches 4 consecutive m/n elements per lane from 4 k-rows: the
// 4 k-rows of one read then fall in 4 distinct granules of a 256-byte bank
// window.
LayoutP tr_lds(i64 rows, i64 k) {
  LayoutP base = make_orderby(make_groupby({rows, k}), {make_regp({rows, k}, {2, 1})});
  if (rows % 32 == 0 && pow2(rows / 32) && rows / 32 >= 2)
    return make_orderby(base, {make_genp(GEN_XOR_SWIZZLE, {k, rows}, {32, 1})});
  return base;
}

// LDS tile for an operand stored in Z order (Morton), whose 16-byte global
// vectors are 2 x 4 blocks of the tile with element bits (k, m, k): each block
// keeps one 16-byte LDS slot in its global order, so it is copied unchanged,
// and the slots of block row r are XOR-permuted by r (a GenP over
// [rows/2, k/4]): the 16 blocks of rows 0-31 at one k, which one half of a
// wave's fragment read touches, fall in 16 distinct granules of a 256-byte
// bank window.  As a layout: TileOrderBy(XOR[rows/2, k/4], Col[2, 2], Row[1, 2]).
LayoutP z_lds(i64 rows, i64 k) {
  return make_tileorderby({make_genp(GEN_XOR_SWIZZLE, {rows / 2, k / 4}, {1, 1}), make_col({2, 2}), make_row({1, 2})});
}

void need_dims(const LayoutP& l, std::vector<i64> d, const char* what) {
  if (l->dims() != d) throw std::length_error(std::string(what) + " layout has the wrong logical shape");
  if (l->expand_inner) throw Unsupported(std::string(what) + ": ExpandBy layouts are not supported by the GEMM");
}

// Does `off` (a function of e and other variables) advance by exactly e, with
// the e = 0 offset a multiple of v?
bool contiguous_in(const Sum& off, int e, int v) {
  Sum ep, rest;
  std::vector<int> g = {e};
  if (!split_by(off, g, &ep, &rest)) return false;
  Ctx dummy;
  if (ep.c0 != 0 || ep.t.size() != 1 || ep.t[0].c != 1) return false;
  const Atom& a = *ep.t[0].a;
  if (a.op != Op::Field || a.var != e || a.a != 1 || a.b != 0) return false;
  return known_multiple(rest) % v == 0;
}

struct Operand {
  // tile [R, KD]: R along m (A) or n (B), KD along k
  i64 R, KD;
  LayoutP glob, lds;
  bool is_b;
  int V = 1, axis = 1, NV = 1;
  int gaxis = 1;  // axis of the widest contiguous global vector (reported)
  // axis 2: a load vector is a VR x VC block of the tile whose V = VR * VC
  // elements are contiguous in global memory in the order given per bit of the
  // element index e: bit b moves by (bdi[b], bdj[b]) (e.g. 2 x 4 blocks of Z order).
  int VR = 1, VC = 1;
  std::vector<i64> bdi, bdj;
  i64 NVEC = 0;
  bool guard = false, sep = false, svec = false, frvec = false;
  bool frtr = false;      // fragments read with the transposing LDS load
  bool frdw = false;      // fragments read as 4 dwords of 2 consecutive k each
  i64 frdw_d = 0;         // element distance of dwords 2h and 2h + 1 (0: not constant)
  bool mpair = false;     // MFMA blocks 2m, 2m+1 take the even / odd rows of a 2*MB band (A only)
  bool frzp = false;      // with mpair: both fragments from two 16-byte reads of 2 x 4 blocks
  i64 rows_total = 0;     // M (A) or N (B): logical extent along the tile rows
  bool edge = false;      // some loads fall outside the operand (padded tiles)
  bool user_lds = false;  // LDS layout given by the caller
  bool direct = false;  // load vector q fills LDS slot q (direct global-to-LDS copy)
};

}  // namespace

namespace {

// `wide_waves`: the default wave tile of a 256-wide workgroup tile is 128
// wide (else 64) along n.
GemmPlan plan_gemm_waves(const GemmRequest& rq0, bool wide_waves) {
  GemmRequest rq = rq0;
  if (rq.dtype != LEGO_F16 && rq.dtype != LEGO_BF16) throw std::invalid_argument("GEMM inputs must be fp16 or bf16");
  if (rq.M <= 0 || rq.N <= 0 || rq.K <= 0) throw std::invalid_argument("GEMM sizes must be positive");
  // Default tiles: 64, 128 or 256 rows (the smallest covering the extent, at
  // most 256), 64-deep k-steps (32 for K < 64); extents they do not divide get
  // padded tiles.
  auto pick = [](i64 n) {
    i64 t = 64;
    while (t < 256 && t < n) t *= 2;
    return (int)t;
  };
  if (!rq.bm) rq.bm = pick(rq.M);
  if (!rq.bn) rq.bn = pick(rq.N);
  if (!rq.bk) rq.bk = rq.K >= 64 ? 64 : 32;
  // Default wave tiles: half the workgroup tile each way (2x2 waves), but at
  // most 64 wide along n for a 256-wide tile unless `wide_waves` (then 128x128
  // wave tiles whose 256 fp32 accumulators fill the AGPRs, one wave per SIMD).
  if (!rq.wm) rq.wm = rq.bm >= 64 ? rq.bm / 2 : rq.bm;
  if (!rq.wn) rq.wn = rq.bn >= 256 && !wide_waves ? 64 : (rq.bn >= 64 ? rq.bn / 2 : rq.bn);
  if (!rq.group_m) rq.group_m = 8;
  const i64 M = rq.M, N = rq.N, K = rq.K;
  const int bm = rq.bm, bn = rq.bn, bk = rq.bk, wm = rq.wm, wn = rq.wn;
  if (bm <= 0 || bn <= 0 || bk <= 0 || wm <= 0 || wn <= 0) throw std::invalid_argument("tile sizes must be positive");
  // Sizes the tiles do not divide are padded to whole tiles (the partial tiles
  // of Section III-D): loads outside [M, K] / [K, N] read zero, stores outside
  // [M, N] are dropped.
  const bool edge_m = M % bm != 0, edge_n = N % bn != 0, edge_k = K % bk != 0;
  int MB = (wm % 32 == 0 && wn % 32 == 0) ? 32 : 16;
  MB = tune("gemm.mfma", MB) == 16 ? 16 : MB;
  {
    // Given fragment layouts select the instruction whose fragments they are.
    int want = -1;
    const LayoutP given[3] = {rq.frag_a, rq.frag_b, rq.frag_c};
    for (int op = 0; op < 3; ++op) {
      if (!given[op]) continue;
      int match = -1;
      for (int instr = 0; instr < 2 && match < 0; ++instr)
        if (same_map(*given[op], *mfma_fragment_layout(instr, op))) match = instr;
      if (match < 0) throw Unsupported("fragment layout is not the fragment layout of a supported MFMA instruction");
      if (want >= 0 && want != match) throw Unsupported("fragment layouts of different MFMA instructions");
      want = match;
    }
    if (want >= 0) MB = want == 0 ? 32 : 16;
  }
  const int KB = MB == 32 ? 16 : 32;
  if (wm % MB || wn % MB || bm % wm || bn % wn || bk % KB)
    throw Unsupported("wave tile must be a multiple of the MFMA block and divide the workgroup tile");
  const int NWM = bm / wm, NWN = bn / wn, NWAVES = NWM * NWN, NT = 64 * NWAVES;
  if (NT > 1024) throw Unsupported("more than 16 waves per workgroup");
  const int MI = wm / MB, NI = wn / MB, NREG = MB == 32 ? 16 : 4;
  if (MI * NI * NREG > 256) throw Unsupported("wave tile needs more than 256 accumulator registers");
  const i64 lds_bytes = 2ll * (bm + bn) * bk * 2;
  if (lds_bytes > 160 * 1024) throw Unsupported("two LDS stages exceed 160 KiB");
  const i64 Mt = (M + bm - 1) / bm, Nt = (N + bn - 1) / bn, Kt = (K + bk - 1) / bk, P = Mt * Nt;

  LayoutP LA = rq.a ? rq.a : make_from_piece(make_row({M, K}));
  LayoutP LB = rq.b ? rq.b : make_from_piece(make_col({K, N}));
  LayoutP LC = rq.c ? rq.c : make_from_piece(make_row({M, N}));
  need_dims(LA, {M, K}, "A");
  need_dims(LB, {K, N}, "B");
  need_dims(LC, {M, N}, "C");
  const i64 G = std::min<i64>(rq.group_m, Mt);
  LayoutP SCH = rq.sched;
  // Grouped order with a ragged last group (Mt % G rows): the full groups are
  // the layout RegP([Mt/G, G, Nt], [1, 3, 2]); the last Mt % G tile rows form one
  // more group in the same column-major order.
  const bool ragged_groups = !SCH && G > 1 && Mt % G != 0;
  if (!SCH) {
    if (Mt % G == 0 && G > 1)
      SCH = make_orderby(make_groupby({Mt, Nt}), {make_regp({Mt / G, G, Nt}, {1, 3, 2})});
    else if (ragged_groups && Mt / G > 0)
      SCH = make_orderby(make_groupby({Mt / G * G, Nt}), {make_regp({Mt / G, G, Nt}, {1, 3, 2})});
    else
      SCH = make_from_piece(make_row({Mt, Nt}));
  }
  if (!ragged_groups) need_dims(SCH, {Mt, Nt}, "schedule");
  const bool xcd = rq.xcd && P % 8 == 0;
  LayoutP XCD = xcd ? make_orderby(make_groupby({P / 8, 8}), {make_regp({P / 8, 8}, {2, 1})}) : nullptr;
  LayoutP SA = rq.lds_a ? rq.lds_a : default_lds(bm, bk);
  LayoutP SB = rq.lds_b ? rq.lds_b : default_lds(bn, bk);
  need_dims(SA, {bm, bk}, "LDS A");
  need_dims(SB, {bn, bk}, "LDS B");
  LayoutP FA = mfma_fragment_layout(MB == 32 ? 0 : 1, 0);
  LayoutP FC = mfma_fragment_layout(MB == 32 ? 0 : 1, 2);

  // Row of fragment row r of MFMA block mi inside the wave tile: block mi
  // covers rows mi*MB .. mi*MB+MB-1, or with row pairs (mpair) blocks 2m and
  // 2m+1 take the even and the odd rows of rows 2m*MB .. 2m*MB+2MB-1, so that
  // one lane holds two adjacent rows (the two rows of a Z-order block).
  auto wrow = [&](Ctx& c, bool mpair, const Sum& mi, const Sum& r) -> Sum {
    if (mpair) return add(c, add(c, mulc(c, fdiv(c, mi, 2), 2 * MB), mulc(c, r, 2)), fmod(c, mi, 2));
    return add(c, mulc(c, mi, MB), r);
  };
  // How a wave reads its MFMA fragments of operand `o` from its LDS layout:
  // one 16-byte vector per lane, the transposing load, 4 dwords of two
  // consecutive k each, or element by element.
  auto frag_modes = [&](Operand& o) {
    o.frvec = o.frtr = o.frdw = o.frzp = false;
    if (o.mpair) {
      // Row pairs: a lane's fragments of blocks 2m and 2m+1 (rows 2r and
      // 2r+1) from two 16-byte reads (h = 0, 1): element e = 4h + 2t + q of
      // block 2m + p lies at read h's offset + 4t + 2p + q, the offset a
      // multiple of 8 (a 2 x 4 Z block per 16-byte slot).
      Ctx c;
      int lane = c.var("lane", 64), w = c.var("w", NWAVES), m = c.var("m", MI / 2), pp = c.var("p", 2),
          s = c.var("s", bk / KB), h = c.var("h", 2), t = c.var("t", 2), q = c.var("q", 2);
      SymAlg al{&c};
      Sum mi = add(c, mulc(c, var(c, m), 2), var(c, pp));
      Sum e = add(c, add(c, mulc(c, var(c, h), 4), mulc(c, var(c, t), 2)), var(c, q));
      Sum f = FA->apply(al, {var(c, lane), e});
      Sum r = fdiv(c, f, KB), k = fmod(c, f, KB);
      Sum wpos = fdiv(c, var(c, w), NWN);
      Sum row = add(c, mulc(c, wpos, wm), wrow(c, true, mi, r));
      Sum kk = add(c, mulc(c, var(c, s), KB), k);
      const Sum off = o.lds->apply(al, {row, kk});
      Sum dep, rest;
      if (split_by(off, {q, pp, t}, &dep, &rest) && dep.c0 == 0 && dep.t.size() == 3 &&
          known_multiple(rest) % 8 == 0) {
        bool ok = true;
        for (const Term& tm : dep.t) {
          const Atom& a = *tm.a;
          const i64 want = a.var == q ? 1 : (a.var == pp ? 2 : 4);
          ok = ok && a.op == Op::Field && a.a == 1 && a.b == 0 && (a.var == q || a.var == pp || a.var == t) &&
               tm.c == want;
        }
        o.frzp = ok;
      }
      return;
    }
    // Vector fragment read?
    {
      Ctx c;
      int lane = c.var("lane", 64), w = c.var("w", NWAVES), mi = c.var("mi", o.is_b ? NI : MI),
          s = c.var("s", bk / KB), e = c.var("e", 8);
      SymAlg al{&c};
      Sum f = FA->apply(al, {var(c, lane), var(c, e)});
      Sum r = fdiv(c, f, KB), k = fmod(c, f, KB);
      Sum wpos = o.is_b ? fmod(c, var(c, w), NWN) : fdiv(c, var(c, w), NWN);
      Sum row = add(c, mulc(c, wpos, o.is_b ? wn : wm), wrow(c, o.mpair, var(c, mi), r));
      Sum kk = add(c, mulc(c, var(c, s), KB), k);
      o.frvec = contiguous_in(o.lds->apply(al, {row, kk}), e, 8);
    }
    // Transposing fragment read (ds_read_b64_tr_b16): in each 16-lane block b,
    // lane i receives element j from the address of lane 16b + 4j + i/4 plus
    // i%4.  It serves a fragment when 4 lanes 4q..4q+3 of a block hold 4
    // consecutive rows at equal k (checked on the fragment layout) and 4
    // consecutive rows are 4 contiguous LDS elements, 4-aligned (checked on
    // the LDS layout).
    if (!o.frvec) {
      IntAlg ia;
      bool lanes_ok = true;
      for (i64 l0 = 0; l0 < 64 && lanes_ok; l0 += 4)
        for (i64 e = 0; e < 8 && lanes_ok; ++e) {
          i64 f0 = FA->apply(ia, {l0, e});
          for (i64 t = 1; t < 4; ++t)
            if (FA->apply(ia, {l0 + t, e}) != f0 + t * KB) lanes_ok = false;
        }
      Ctx c;
      int w = c.var("w", NWAVES), mi = c.var("mi", o.is_b ? NI : MI), rr = c.var("rr", MB / 4),
          kq = c.var("kq", bk), t = c.var("t", 4);
      SymAlg al{&c};
      Sum wpos = o.is_b ? fmod(c, var(c, w), NWN) : fdiv(c, var(c, w), NWN);
      Sum row = add(c, add(c, mulc(c, wpos, o.is_b ? wn : wm), mulc(c, var(c, mi), MB)),
                    add(c, mulc(c, var(c, rr), 4), var(c, t)));
      o.frtr = lanes_ok && contiguous_in(o.lds->apply(al, {row, var(c, kq)}), t, 4);
    }
    // Dword reads: fragment elements 2p and 2p + 1 adjacent in LDS, the pair
    // 4-byte aligned (p = 2h + t).  When the offset moves by a constant D
    // from t = 0 to t = 1, each half h is one address and the read pairs
    // (that address, + D) become single ds_read2_b32 instructions.
    if (!o.frvec && !o.frtr) {
      Ctx c;
      int lane = c.var("lane", 64), w = c.var("w", NWAVES), mi = c.var("mi", o.is_b ? NI : MI),
          s = c.var("s", bk / KB), h = c.var("h", 2), t = c.var("t", 2), q = c.var("q", 2);
      SymAlg al{&c};
      Sum e = add(c, add(c, mulc(c, var(c, h), 4), mulc(c, var(c, t), 2)), var(c, q));
      Sum f = FA->apply(al, {var(c, lane), e});
      Sum r = fdiv(c, f, KB), k = fmod(c, f, KB);
      Sum wpos = o.is_b ? fmod(c, var(c, w), NWN) : fdiv(c, var(c, w), NWN);
      Sum row = add(c, mulc(c, wpos, o.is_b ? wn : wm), wrow(c, o.mpair, var(c, mi), r));
      Sum kk = add(c, mulc(c, var(c, s), KB), k);
      const Sum off = o.lds->apply(al, {row, kk});
      o.frdw = contiguous_in(off, q, 2);
      o.frdw_d = 0;
      Sum pt, rest;
      std::vector<int> g = {t};
      if (o.frdw && split_by(off, g, &pt, &rest) && pt.c0 == 0 && pt.t.size() == 1) {
        const Atom& a = *pt.t[0].a;
        if (a.op == Op::Field && a.var == t && a.a == 1 && a.b == 0 && pt.t[0].c > 0 && pt.t[0].c % 2 == 0)
          o.frdw_d = pt.t[0].c;
      }
    }
  };

  Operand ops[2] = {{bm, bk, LA, SA, false}, {bn, bk, LB, SB, true}};
  ops[0].user_lds = (bool)rq.lds_a;
  ops[1].user_lds = (bool)rq.lds_b;
  ops[0].rows_total = M;
  ops[1].rows_total = N;
  ops[0].edge = edge_m || edge_k;
  ops[1].edge = edge_n || edge_k;
  // Validity of tile element (i, j) at tile coordinates (tt, kt): inside the
  // operand's logical extents.
  auto in_range = [&](Ctx& c, const Operand& o, const Sum& tt, const Sum& kt, const Sum& i, const Sum& j) {
    Sum row = add(c, mulc(c, tt, o.R), i);
    Sum kk = add(c, mulc(c, kt, o.KD), j);
    return mul(c, lt(c, row, cst(o.rows_total)), lt(c, kk, cst(K)));
  };
  // With a single round of load vectors, only threads below NVEC load; giving
  // tid that range lets the range analysis prove separability.
  auto tid_ext = [&](const Operand& o) -> i64 { return o.NV == 1 ? std::min<i64>(NT, o.NVEC) : NT; };

  // Global element offset of tile element (i, j) for tile coordinates (tt, kt).
  auto glob_off = [&](Ctx& c, const Operand& o, const Sum& tt, const Sum& kt, const Sum& i, const Sum& j) {
    SymAlg al{&c};
    Sum row = add(c, mulc(c, tt, o.R), i);
    Sum kk = add(c, mulc(c, kt, o.KD), j);
    return o.is_b ? o.glob->apply(al, {kk, row}) : o.glob->apply(al, {row, kk});
  };
  // Tile element (i, j) of load vector u of thread tid, plus element e.
  auto load_elem = [&](Ctx& c, const Operand& o, const Sum& tid, const Sum& u, const Sum& e, Sum* i, Sum* j) {
    Sum q = add(c, mulc(c, u, NT), tid);
    if (o.direct) {
      // Slot q of the LDS tile holds the elements S^{-1}(8q + e).
      SymAlg al{&c};
      std::vector<Sum> ij = o.lds->inv(al, add(c, mulc(c, q, 8), e));
      *i = ij[0];
      *j = ij[1];
      return;
    }
    if (o.axis == 2) {
      i64 per = o.KD / o.VC;
      Sum di = cst(0), dj = cst(0);
      for (size_t b = 0; b < o.bdi.size(); ++b) {
        Sum bit = fmod(c, fdiv(c, e, i64(1) << b), 2);
        di = add(c, di, mulc(c, bit, o.bdi[b]));
        dj = add(c, dj, mulc(c, bit, o.bdj[b]));
      }
      *i = add(c, mulc(c, fdiv(c, q, per), o.VR), di);
      *j = add(c, mulc(c, fmod(c, q, per), o.VC), dj);
    } else if (o.axis == 1) {
      i64 per = o.KD / o.V;
      *i = fdiv(c, q, per);
      *j = add(c, mulc(c, fmod(c, q, per), o.V), e);
    } else {
      i64 per = o.R / o.V;
      *i = add(c, mulc(c, fmod(c, q, per), o.V), e);
      *j = fdiv(c, q, per);
    }
  };

  for (Operand& o : ops) {
    // Largest vector (16 bytes at most) along either tile axis that is
    // contiguous and aligned in global memory.
    o.V = 1;
    o.axis = 1;
    for (int v : {8, 4, 2}) {
      bool found = false;
      for (int axis : {1, 0}) {
        i64 ext = axis == 1 ? o.KD : o.R;
        if (ext % v) continue;
        Ctx c;
        int tt = c.var("tt", o.is_b ? Nt : Mt), kt = c.var("kt", Kt);
        int x = c.var("x", ext / v), y = c.var("y", axis == 1 ? o.R : o.KD), e = c.var("e", v);
        Sum xs = add(c, mulc(c, var(c, x), v), var(c, e));
        Sum off = axis == 1 ? glob_off(c, o, var(c, tt), var(c, kt), var(c, y), xs)
                            : glob_off(c, o, var(c, tt), var(c, kt), xs, var(c, y));
        // With padded tiles a vector must lie wholly inside or wholly outside.
        Sum ok = axis == 1 ? in_range(c, o, var(c, tt), var(c, kt), var(c, y), xs)
                           : in_range(c, o, var(c, tt), var(c, kt), xs, var(c, y));
        if (contiguous_in(off, e, v) && !(o.edge && depends_on(ok, e))) {
          o.V = v;
          o.axis = axis;
          found = true;
          break;
        }
      }
      if (found) break;
    }
    // No 16-byte run along one axis: try 8 elements contiguous in global memory
    // that form a small 2D block of the tile (Z order keeps 2 x 4 blocks together).
    if (o.V < 8) {
      for (auto shape : {std::pair<int, int>{2, 4}, {4, 2}}) {
        const int vr = shape.first, vc = shape.second;
        if (o.R % vr || o.KD % vc) continue;
        // The order of the 8 elements, read off the layout at the origin.
        IntAlg ia;
        const i64 g0 = o.is_b ? o.glob->apply(ia, {0, 0}) : o.glob->apply(ia, {0, 0});
        std::vector<i64> di(8), dj(8);
        bool ok = true;
        for (int e = 0; e < 8 && ok; ++e) {
          if (g0 + e >= o.glob->phys_size()) {
            ok = false;
            break;
          }
          std::vector<i64> lc = o.glob->inv(ia, g0 + e);
          di[e] = o.is_b ? lc[1] : lc[0];
          dj[e] = o.is_b ? lc[0] : lc[1];
          ok = di[e] >= 0 && di[e] < vr && dj[e] >= 0 && dj[e] < vc;
        }
        // linear over the bits of e
        for (int e = 0; e < 8 && ok; ++e) {
          i64 si = 0, sj = 0;
          for (int b = 0; b < 3; ++b)
            if (e >> b & 1) si += di[1 << b], sj += dj[1 << b];
          ok = si == di[e] && sj == dj[e];
        }
        if (!ok) continue;
        Operand t = o;
        t.axis = 2;
        t.V = 8;
        t.VR = vr;
        t.VC = vc;
        t.bdi = {di[1], di[2], di[4]};
        t.bdj = {dj[1], dj[2], dj[4]};
        // every block of every tile: 8 contiguous, aligned elements
        Ctx c;
        int tt = c.var("tt", o.is_b ? Nt : Mt), kt = c.var("kt", Kt), q = c.var("q", o.R * o.KD / 8),
            e = c.var("e", 8);
        Sum i, j;
        load_elem(c, t, var(c, q), cst(0), var(c, e), &i, &j);
        Sum off = glob_off(c, t, var(c, tt), var(c, kt), i, j);
        Sum okv = in_range(c, t, var(c, tt), var(c, kt), i, j);
        if (contiguous_in(off, e, 8) && !(o.edge && depends_on(okv, e))) {
          o = t;
          break;
        }
      }
    }
    o.gaxis = o.axis;
    // An operand contiguous along m/n keeps that orientation in LDS.
    if (!o.user_lds && o.axis == 0 && o.V >= 4) o.lds = tr_lds(o.R, o.KD);
    o.NVEC = o.R * o.KD / o.V;
    o.NV = (int)((o.NVEC + NT - 1) / NT);
    o.guard = o.NVEC % NT != 0;
    // Additive separability of the global offset into tile, k-step and thread parts.
    {
      Ctx c;
      int tt = c.var("tt", o.is_b ? Nt : Mt), kt = c.var("kt", Kt), tid = c.var("tid", tid_ext(o)),
          u = c.var("u", o.NV);
      Sum i, j;
      load_elem(c, o, var(c, tid), var(c, u), cst(0), &i, &j);
      Sum off = glob_off(c, o, var(c, tt), var(c, kt), i, j);
      Sum pt, r1, pk, pl;
      o.sep = split_by(off, {tt}, &pt, &r1) && split_by(r1, {kt}, &pk, &pl);
    }
    // Vector LDS store?
    {
      Ctx c;
      int tid = c.var("tid", tid_ext(o)), u = c.var("u", o.NV), e = c.var("e", o.V);
      Sum i, j;
      load_elem(c, o, var(c, tid), var(c, u), var(c, e), &i, &j);
      SymAlg al{&c};
      if (o.axis == 2) {
        // stored one block row at a time: VC elements contiguous in LDS
        Sum i0, j0;
        load_elem(c, o, var(c, tid), var(c, u), cst(0), &i0, &j0);
        int r = c.var("r", o.VR), cc = c.var("cc", o.VC);
        o.svec = contiguous_in(o.lds->apply(al, {add(c, i0, var(c, r)), add(c, j0, var(c, cc))}), cc, o.VC);
      } else {
        o.svec = o.V > 1 && contiguous_in(o.lds->apply(al, {i, j}), e, o.V);
        if (o.V == 1) o.svec = true;
      }
    }
    frag_modes(o);
  }

  // Z-order operands (2 x 4 blocks with element bits k, m, k) can be copied
  // directly into the z_lds layout, which keeps each block in one LDS slot;
  // a lane then reads its row's 8 k as 4 dwords (2 k each).
  LayoutP zl[2];
  bool zpair[2] = {false, false};
  for (int k = 0; k < 2; ++k) {
    const Operand& o = ops[k];
    if (o.user_lds || o.axis != 2 || o.VR != 2 || o.VC != 4 || o.bdi != std::vector<i64>{0, 1, 0} ||
        o.bdj != std::vector<i64>{1, 0, 2} || o.R % 2 || o.KD % 8 || !pow2(o.KD / 4) || !tune("gemm.zdirect", 1))
      continue;
    Operand t = o;
    t.lds = z_lds(o.R, o.KD);
    if (!o.is_b && MI % 2 == 0 && tune("gemm.zpair", 1)) {
      t.mpair = true;
      frag_modes(t);
      if (t.frzp) {
        zl[k] = t.lds;
        zpair[k] = true;
        continue;
      }
      t.mpair = false;
    }
    frag_modes(t);
    if (t.frdw) zl[k] = t.lds;
  }
  // Direct global-to-LDS copies need 16-byte global runs under the inverse
  // LDS layout and whole rounds of load vectors.
  bool direct = true;
  direct = tune("gemm.direct", 1) != 0;
  if ((bk / KB) % 2) direct = false;  // the direct loop alternates fragment buffers per substep
  for (int k = 0; k < 2; ++k) {
    const Operand& o = ops[k];
    if (!direct) break;
    if ((o.R * o.KD) % (8 * NT)) {
      direct = false;
      break;
    }
    Operand t = o;
    t.direct = true;
    if (zl[k]) t.lds = zl[k];
    t.V = 8;
    t.NV = (int)(o.R * o.KD / 8 / NT);
    Ctx c;
    int tt = c.var("tt", o.is_b ? Nt : Mt), kt = c.var("kt", Kt), tid = c.var("tid", NT), u = c.var("u", t.NV),
        e = c.var("e", 8);
    Sum i, j;
    load_elem(c, t, var(c, tid), var(c, u), var(c, e), &i, &j);
    if (!contiguous_in(glob_off(c, t, var(c, tt), var(c, kt), i, j), e, 8)) direct = false;
    // Padded tiles: whole-vector validity, and 32-bit byte offsets for the
    // range-checked buffer loads that fill out-of-range slots with zero.
    if (o.edge && (depends_on(in_range(c, t, var(c, tt), var(c, kt), i, j), e) ||
                   2 * o.glob->phys_size() >= (i64(1) << 31)))
      direct = false;
  }
  if (direct) {
    for (int k = 0; k < 2; ++k) {
      Operand& o = ops[k];
      if (zl[k]) {
        o.lds = zl[k];
        o.mpair = zpair[k];
        frag_modes(o);
      }
      o.direct = true;
      o.V = 8;
      o.axis = 1;
      o.NVEC = o.R * o.KD / 8;
      o.NV = (int)(o.NVEC / NT);
      o.guard = false;
      o.svec = true;
      Ctx c;
      int tt = c.var("tt", o.is_b ? Nt : Mt), kt = c.var("kt", Kt), tid = c.var("tid", NT), u = c.var("u", o.NV);
      Sum i, j;
      load_elem(c, o, var(c, tid), var(c, u), cst(0), &i, &j);
      Sum off = glob_off(c, o, var(c, tt), var(c, kt), i, j);
      Sum pt, r1, pk, pl;
      o.sep = split_by(off, {tt}, &pt, &r1) && split_by(r1, {kt}, &pk, &pl);
    }
  }
  const i64 stage_bytes = 2ll * (bm + bn) * bk;
  int nstages = 2;
  if (direct) {
    nstages = (int)std::min<i64>(4, (160 * 1024) / stage_bytes);
    // the waits count loads: NSTAGES-1 tiles behind the awaited one must fit vmcnt's 63
    const i64 per_tile = ops[0].NV + ops[1].NV;
    while (nstages > 2 && (nstages - 1) * per_tile > 63) --nstages;
    if (per_tile > 63) direct = false;
    if (rq.stages) {
      if (rq.stages < 2 || rq.stages > 4 || rq.stages * stage_bytes > 160 * 1024 || (rq.stages - 1) * per_tile > 63)
        throw Unsupported("this many LDS stages do not fit the LDS or the load counter");
      nstages = rq.stages;
    }
  }
  // Register-staged plans double-buffer the LDS tile.
  if (!direct && rq.stages && rq.stages != 2) throw Unsupported("register-staged plans use two LDS stages");

  // ----- emit the index functions
  using Builder = std::function<FnSpec(Ctx&)>;
  std::vector<std::pair<std::string, Builder>> fns;
  // Parts of one additive split (a_gt/a_gk/a_gl, b_*, c_t/c_l) are all taken
  // from the expanded lowering, the one the separability check used.
  auto is_part = [](const std::string& n) {
    return n == "a_gt" || n == "a_gk" || n == "a_gl" || n == "b_gt" || n == "b_gk" || n == "b_gl" || n == "c_t" ||
           n == "c_l";
  };
  fns.push_back({"sched", [&](Ctx& c) {
                   SymAlg al{&c};
                   int pid = c.var("pid", P);
                   Sum q = var(c, pid);
                   if (xcd) q = XCD->apply(al, unflatten(al, {P / 8, 8}, q));
                   FnSpec f;
                   f.params = {pid};
                   if (!ragged_groups) {
                     f.outs = SCH->inv(al, q);
                     return f;
                   }
                   // Full groups first, then the ragged group of r = Mt % G rows.
                   const i64 full = Mt / G * G, r = Mt % G, nfull = full * Nt;
                   Sum rest = sub(c, q, cst(nfull));
                   Sum tm_r = add(c, cst(full), fmod(c, rest, r)), tn_r = fdiv(c, rest, r);
                   if (full == 0) {
                     f.outs = {tm_r, tn_r};
                     return f;
                   }
                   Sum in_full = lt(c, q, cst(nfull));
                   // Clamp the argument of the full-group layout into its domain.
                   Sum qf = select(c, in_full, q, cst(0));
                   std::vector<Sum> g = SCH->inv(al, qf);
                   f.outs = {select(c, in_full, g[0], tm_r), select(c, in_full, g[1], tn_r)};
                   return f;
                 }});
  const char* pre[2] = {"a_", "b_"};
  for (int k = 0; k < 2; ++k) {
    const Operand& o = ops[k];
    std::string p = pre[k];
    auto full = [&, k](Ctx& c, int* tt, int* kt, int* tid, int* u) {
      const Operand& oo = ops[k];
      *tt = c.var(oo.is_b ? "tn" : "tm", oo.is_b ? Nt : Mt);
      *kt = c.var("kt", Kt);
      *tid = c.var("tid", tid_ext(oo));
      *u = c.var("u", oo.NV);
      Sum i, j;
      load_elem(c, oo, var(c, *tid), var(c, *u), cst(0), &i, &j);
      return glob_off(c, oo, var(c, *tt), var(c, *kt), i, j);
    };
    if (o.sep) {
      fns.push_back({p + "gt", [=](Ctx& c) {
                       int tt, kt, tid, u;
                       Sum off = full(c, &tt, &kt, &tid, &u), a, r;
                       FnSpec f;
                       f.valid = split_by(off, {tt}, &a, &r);
                       f.params = {tt};
                       f.outs = {a};
                       return f;
                     }});
      fns.push_back({p + "gk", [=](Ctx& c) {
                       int tt, kt, tid, u;
                       Sum off = full(c, &tt, &kt, &tid, &u), a, r, kp, l;
                       FnSpec f;
                       f.valid = split_by(off, {tt}, &a, &r) && split_by(r, {kt}, &kp, &l);
                       f.params = {kt};
                       f.outs = {kp};
                       return f;
                     }});
      fns.push_back({p + "gl", [=](Ctx& c) {
                       int tt, kt, tid, u;
                       Sum off = full(c, &tt, &kt, &tid, &u), a, r, kp, l;
                       FnSpec f;
                       f.valid = split_by(off, {tt}, &a, &r) && split_by(r, {kt}, &kp, &l);
                       f.params = {tid, u};
                       f.outs = {l};
                       return f;
                     }});
    } else {
      fns.push_back({p + "gf", [=](Ctx& c) {
                       int tt, kt, tid, u;
                       Sum off = full(c, &tt, &kt, &tid, &u);
                       FnSpec f;
                       f.params = {tt, kt, tid, u};
                       f.outs = {off};
                       return f;
                     }});
    }
    fns.push_back({p + "s", [&, k](Ctx& c) {
                     const Operand& oo = ops[k];
                     int tid = c.var("tid", tid_ext(oo)), u = c.var("u", oo.NV), e = c.var("e", oo.V);
                     Sum i, j;
                     load_elem(c, oo, var(c, tid), var(c, u), var(c, e), &i, &j);
                     SymAlg al{&c};
                     FnSpec f;
                     f.params = {tid, u, e};
                     f.outs = {oo.lds->apply(al, {i, j})};
                     return f;
                   }});
    fns.push_back({p + "fr", [&, k](Ctx& c) {
                     const Operand& oo = ops[k];
                     int lane = c.var("lane", 64), w = c.var("w", NWAVES), mi = c.var("mi", oo.is_b ? NI : MI),
                         s = c.var("s", bk / KB), e = c.var("e", 8);
                     SymAlg al{&c};
                     Sum f0 = FA->apply(al, {var(c, lane), var(c, e)});
                     Sum r = fdiv(c, f0, KB), kq = fmod(c, f0, KB);
                     Sum wpos = oo.is_b ? fmod(c, var(c, w), NWN) : fdiv(c, var(c, w), NWN);
                     Sum row = add(c, mulc(c, wpos, oo.is_b ? wn : wm), wrow(c, oo.mpair, var(c, mi), r));
                     Sum kk = add(c, mulc(c, var(c, s), KB), kq);
                     FnSpec f;
                     f.params = {lane, w, mi, s, e};
                     f.outs = {oo.lds->apply(al, {row, kk})};
                     return f;
                   }});
    if (o.edge)
      fns.push_back({p + "ok", [&, k](Ctx& c) {
                       // 1 when load vector u of thread tid at tile (tt, kt) lies
                       // inside the operand, 0 when it is padding.
                       const Operand& oo = ops[k];
                       int tt = c.var(oo.is_b ? "tn" : "tm", oo.is_b ? Nt : Mt), kt = c.var("kt", Kt),
                           tid = c.var("tid", tid_ext(oo)), u = c.var("u", oo.NV);
                       Sum i, j;
                       load_elem(c, oo, var(c, tid), var(c, u), cst(0), &i, &j);
                       FnSpec f;
                       f.params = {tt, kt, tid, u};
                       f.outs = {in_range(c, oo, var(c, tt), var(c, kt), i, j)};
                       return f;
                     }});
    if (o.frzp)
      fns.push_back({p + "fz", [&, k](Ctx& c) {
                       // LDS offset of the 16-byte read h of the fragment pair
                       // (blocks 2m, 2m+1): fragment element 4h of block 2m.
                       const Operand& oo = ops[k];
                       int lane = c.var("lane", 64), w = c.var("w", NWAVES), m = c.var("m", MI / 2),
                           s = c.var("s", bk / KB), h = c.var("h", 2);
                       SymAlg al{&c};
                       Sum f0 = FA->apply(al, {var(c, lane), mulc(c, var(c, h), 4)});
                       Sum r = fdiv(c, f0, KB), kq = fmod(c, f0, KB);
                       Sum wpos = fdiv(c, var(c, w), NWN);
                       Sum row = add(c, mulc(c, wpos, wm), wrow(c, true, mulc(c, var(c, m), 2), r));
                       Sum kk = add(c, mulc(c, var(c, s), KB), kq);
                       FnSpec f;
                       f.params = {lane, w, m, s, h};
                       f.outs = {oo.lds->apply(al, {row, kk})};
                       return f;
                     }});
    if (o.frdw && o.frdw_d)
      fns.push_back({p + "fd", [&, k](Ctx& c) {
                       // LDS offset of fragment element 4h: the first dword of
                       // half h (the second lies FRDW_D elements further).
                       const Operand& oo = ops[k];
                       int lane = c.var("lane", 64), w = c.var("w", NWAVES), mi = c.var("mi", oo.is_b ? NI : MI),
                           s = c.var("s", bk / KB), h = c.var("h", 2);
                       SymAlg al{&c};
                       Sum f0 = FA->apply(al, {var(c, lane), mulc(c, var(c, h), 4)});
                       Sum r = fdiv(c, f0, KB), kq = fmod(c, f0, KB);
                       Sum wpos = oo.is_b ? fmod(c, var(c, w), NWN) : fdiv(c, var(c, w), NWN);
                       Sum row = add(c, mulc(c, wpos, oo.is_b ? wn : wm), wrow(c, oo.mpair, var(c, mi), r));
                       Sum kk = add(c, mulc(c, var(c, s), KB), kq);
                       FnSpec f;
                       f.params = {lane, w, mi, s, h};
                       f.outs = {oo.lds->apply(al, {row, kk})};
                       return f;
                     }});
    if (o.frtr)
      fns.push_back({p + "ft", [&, k](Ctx& c) {
                       // Address lane `lane` supplies to the transposing read of
                       // half h: the element that lane 16*(lane/16) + 4*(lane%4)
                       // needs at fragment element 4h + (lane%16)/4.
                       const Operand& oo = ops[k];
                       int lane = c.var("lane", 64), w = c.var("w", NWAVES), mi = c.var("mi", oo.is_b ? NI : MI),
                           s = c.var("s", bk / KB), h = c.var("h", 2);
                       SymAlg al{&c};
                       Sum lp = add(c, mulc(c, fdiv(c, var(c, lane), 16), 16), mulc(c, fmod(c, var(c, lane), 4), 4));
                       Sum ep = add(c, mulc(c, var(c, h), 4), fdiv(c, fmod(c, var(c, lane), 16), 4));
                       Sum f0 = FA->apply(al, {lp, ep});
                       Sum r = fdiv(c, f0, KB), kq = fmod(c, f0, KB);
                       Sum wpos = oo.is_b ? fmod(c, var(c, w), NWN) : fdiv(c, var(c, w), NWN);
                       Sum row = add(c, mulc(c, wpos, oo.is_b ? wn : wm), wrow(c, oo.mpair, var(c, mi), r));
                       Sum kk = add(c, mulc(c, var(c, s), KB), kq);
                       FnSpec f;
                       f.params = {lane, w, mi, s, h};
                       f.outs = {oo.lds->apply(al, {row, kk})};
                       return f;
                     }});
  }
  auto c_full = [&](Ctx& c, int* tm, int* tn, int* lane, int* w, int* mi, int* ni, int* r) {
    *tm = c.var("tm", Mt);
    *tn = c.var("tn", Nt);
    *lane = c.var("lane", 64);
    *w = c.var("w", NWAVES);
    *mi = c.var("mi", MI);
    *ni = c.var("ni", NI);
    *r = c.var("r", NREG);
    SymAlg al{&c};
    Sum f0 = FC->apply(al, {var(c, *lane), var(c, *r)});
    Sum row = fdiv(c, f0, MB), col = fmod(c, f0, MB);
    Sum m = add(c, add(c, mulc(c, var(c, *tm), bm), mulc(c, fdiv(c, var(c, *w), NWN), wm)),
                wrow(c, ops[0].mpair, var(c, *mi), row));
    Sum n = add(c, add(c, mulc(c, var(c, *tn), bn), mulc(c, fmod(c, var(c, *w), NWN), wn)),
                add(c, mulc(c, var(c, *ni), MB), col));
    return LC->apply(al, {m, n});
  };
  const bool cedge = edge_m || edge_n;
  if (cedge)
    fns.push_back({"c_ok", [&](Ctx& c) {
                     int tm = c.var("tm", Mt), tn = c.var("tn", Nt), lane = c.var("lane", 64),
                         w = c.var("w", NWAVES), mi = c.var("mi", MI), ni = c.var("ni", NI), r = c.var("r", NREG);
                     SymAlg al{&c};
                     Sum f0 = FC->apply(al, {var(c, lane), var(c, r)});
                     Sum row = fdiv(c, f0, MB), col = fmod(c, f0, MB);
                     Sum m = add(c, add(c, mulc(c, var(c, tm), bm), mulc(c, fdiv(c, var(c, w), NWN), wm)),
                                 wrow(c, ops[0].mpair, var(c, mi), row));
                     Sum n = add(c, add(c, mulc(c, var(c, tn), bn), mulc(c, fmod(c, var(c, w), NWN), wn)),
                                 add(c, mulc(c, var(c, ni), MB), col));
                     FnSpec f;
                     f.params = {tm, tn, lane, w, mi, ni, r};
                     f.outs = {mul(c, lt(c, m, cst(M)), lt(c, n, cst(N)))};
                     return f;
                   }});
  bool csep = false;
  {
    Ctx c;
    int tm, tn, lane, w, mi, ni, r;
    Sum off = c_full(c, &tm, &tn, &lane, &w, &mi, &ni, &r), a, b;
    csep = split_by(off, {tm, tn}, &a, &b);
  }
  if (csep) {
    fns.push_back({"c_t", [&](Ctx& c) {
                     int tm, tn, lane, w, mi, ni, r;
                     Sum off = c_full(c, &tm, &tn, &lane, &w, &mi, &ni, &r), a, b;
                     FnSpec f;
                     f.valid = split_by(off, {tm, tn}, &a, &b);
                     f.params = {tm, tn};
                     f.outs = {a};
                     return f;
                   }});
    fns.push_back({"c_l", [&](Ctx& c) {
                     int tm, tn, lane, w, mi, ni, r;
                     Sum off = c_full(c, &tm, &tn, &lane, &w, &mi, &ni, &r), a, b;
                     FnSpec f;
                     f.valid = split_by(off, {tm, tn}, &a, &b);
                     f.params = {lane, w, mi, ni, r};
                     f.outs = {b};
                     return f;
                   }});
  } else {
    fns.push_back({"c_f", [&](Ctx& c) {
                     int tm, tn, lane, w, mi, ni, r;
                     Sum off = c_full(c, &tm, &tn, &lane, &w, &mi, &ni, &r);
                     FnSpec f;
                     f.params = {tm, tn, lane, w, mi, ni, r};
                     f.outs = {off};
                     return f;
                   }});
  }

  bool wide = false;
  for (auto& f : fns) wide = wide || emit_best(f.first, f.second, false, is_part(f.first) ? 0 : -1).wide;
  std::string code;
  std::ostringstream opsinfo;
  for (auto& f : fns) {
    Emitted e = emit_best(f.first, f.second, wide, is_part(f.first) ? 0 : -1);
    code += e.code;
    opsinfo << " " << f.first << ":" << e.ops;
  }

  // MFMA blocks of a wave tile with a row (column) inside C in some tile:
  // the first row of block i (column of block j) in the first wave of the
  // first tile is its least, so the blocks with no element in range in any
  // tile are a suffix (M or N below one tile).  Row pairs are read together.
  int mi_live = 0, ni_live = 0;
  for (int i = 0; i < MI; ++i)
    if ((ops[0].mpair ? (i / 2) * 2 * MB + i % 2 : i * MB) < M) mi_live = i + 1;
  if (ops[0].mpair && mi_live % 2) ++mi_live;
  for (int j = 0; j < NI; ++j)
    if (j * MB < N) ni_live = j + 1;

  std::ostringstream s;
  s << prelude_text() << "#define IDX_T " << (wide ? "i64" : "u32") << "\n"
    << "#define MI_LIVE " << mi_live << "\n#define NI_LIVE " << ni_live << "\n"
    << "#define BM " << bm << "\n#define BN " << bn << "\n#define BK " << bk << "\n#define MB " << MB
    << "\n#define KB " << KB << "\n#define MI " << MI << "\n#define NI " << NI << "\n#define NWAVES " << NWAVES
    << "\n#define NT " << NT << "\n#define KT " << Kt << "u\n#define IN_BF16 " << (rq.dtype == LEGO_BF16 ? 1 : 0)
    << "\n#define GEMM_M " << M << "ull\n#define GEMM_N " << N << "ull\n#define GEMM_K " << K << "ull\n#define GEMM_MT "
    << Mt << "ull\n#define GEMM_NT " << Nt << "ull\n";
  const char* P2[2] = {"A_", "B_"};
  for (int k = 0; k < 2; ++k) {
    const Operand& o = ops[k];
    s << "#define " << P2[k] << "NV " << o.NV << "\n#define " << P2[k] << "V " << o.V << "\n#define " << P2[k]
      << "SEP " << (o.sep ? 1 : 0) << "\n#define " << P2[k] << "SVEC " << (o.svec ? 1 : 0) << "\n#define " << P2[k]
      << "FRVEC " << (o.frvec ? 1 : 0) << "\n#define " << P2[k] << "FRTR " << (o.frtr ? 1 : 0) << "\n#define " << P2[k]
      << "FRDW " << (o.frdw ? 1 : 0) << "\n#define " << P2[k] << "FRDW_D " << o.frdw_d << "\n#define " << P2[k]
      << "FRZP " << (o.frzp ? 1 : 0) << "\n#define " << P2[k]
      << "NVEC " << o.NVEC << "u\n#define " << P2[k]
      << "GUARD " << (o.guard ? 1 : 0) << "\n#define " << P2[k] << "EDGE " << (o.edge ? 1 : 0) << "\n#define "
      << P2[k] << "BUF " << (o.direct && 2 * o.glob->phys_size() < (i64(1) << 31) ? 1 : 0) << "\n#define "
      << P2[k] << "BYTES " << 2 * o.glob->phys_size() << "u\n#define " << P2[k] << "VR " << o.VR << "\n#define "
      << P2[k] << "VC " << (o.axis == 2 ? o.VC : o.V) << "\n";
    // Block vectors: element index of block position (r, c), row-major.
    s << "static constexpr int " << P2[k] << "BIDX[] = {";
    if (o.axis == 2) {
      for (int r = 0; r < o.VR; ++r)
        for (int cc = 0; cc < o.VC; ++cc)
          for (int e = 0; e < o.V; ++e) {
            i64 di = 0, dj = 0;
            for (int b = 0; b < 3; ++b)
              if (e >> b & 1) di += o.bdi[b], dj += o.bdj[b];
            if (di == r && dj == cc) s << e << ",";
          }
    } else {
      s << "0";
    }
    s << "};\n";
  }
  s << "#define C_EDGE " << (cedge ? 1 : 0) << "\n";
  // Two staging register sets when the accumulators live in AGPRs (one wave
  // per SIMD leaves the VGPRs for them); one otherwise, so two waves fit.
  int prefetch = (MI * NI * NREG > 128) ? 2 : 1;
  prefetch = tune("gemm.prefetch", prefetch) == 2 ? 2 : 1;
  if (Kt < 2) prefetch = 1;
  // Register-staged plans use the rolling pipeline (one staging set; LDS
  // writes and reloads spread over the substeps): measured +7% on the 8192^3
  // bf16 GEMM and +16% on the 4096^3 Morton-A GEMM over staging the whole
  // tile in one substep.
  int rolling = 1;
  rolling = tune("gemm.rolling", rolling) != 0;
  // The direct copies of the next tile go out between MFMA rows rather than
  // in one burst (measured 0.87 -> 0.85 ms on the 8192^3 bf16 GEMM with
  // 128x128 wave tiles, and 0.870 -> 0.864 ms with 8 waves of 128x64).
  int dma_spread = 1;
  dma_spread = tune("gemm.dma_spread", dma_spread) != 0;
  // Direct-copy plans read fragments two substeps ahead of their MFMAs, so
  // that reads held up by copies landing in LDS do not stall them (0.857 ->
  // 0.852 ms on the 8192^3 bf16 GEMM); not with the transposing reads, whose
  // wait at each substep covers every read in flight.
  int frag_dist = 2;
  frag_dist = (int)std::max<long long>(1, std::min<long long>(3, tune("gemm.frag_dist", frag_dist)));
  // (Reads two substeps ahead need three substeps per step: with two, the
  // early reads of the last substep would replace fragments its later MFMA
  // rows still use.)
  if (!direct || bk / KB <= frag_dist) frag_dist = 1;
  if (const long long rows = tune("gemm.dma_rows", 0)) s << "#define DMA_ROWS " << rows << "\n";
  // Loop unrolled over the LDS ring when one wave per SIMD leaves the
  // registers for per-stage fragment addresses.
  const int ring_unroll = (int)tune("gemm.ring_unroll", MI * NI * NREG > 128 ? 1 : 0);
  s << "#define RING_UNROLL " << ring_unroll << "\n#define FRAG_SPREAD " << tune("gemm.frag_spread", 2) << "\n";
  s << "#define PREFETCH " << prefetch << "\n#define ROLLING " << rolling << "\n#define DMA_SPREAD " << dma_spread
    << "\n#define FRAG_DIST " << frag_dist << "\n#define DIRECT_LDS " << (direct ? 1 : 0)
    << "\n#define NSTAGES " << nstages << "\n";
  int store_at = (int)tune("gemm.store_at", (bk / KB) / 2);
  store_at = std::max(0, std::min(store_at, bk / KB - 1));
  s << "#define STORE_AT " << store_at << "\n";
  // A persistent grid walks several tiles per workgroup, chaining the LDS
  // ring across tiles: the first steps of the next tile are requested during
  // the last NSTAGES steps of the current one, so a tile needs that many.
  // Not with padded tiles: the range checks of two tiles' copies do not fit
  // the registers beside the walk's state (8000^3 bf16: 240 VGPRs spilled
  // with 8 waves, 613 with 4; none without the walk).
  const bool persist = direct && Kt >= nstages && !(ops[0].edge || ops[1].edge || cedge) &&
                       tune("gemm.persist", 1) != 0;
  s << "#define C_SEP " << (csep ? 1 : 0) << "\n#define PERSIST " << (persist ? 1 : 0) << "\n" << code << "// ---- template ----\n" << tpl_gemm;

  GemmPlan g;
  g.src = s.str();
  g.kernel = "lego_gemm";
  g.grid = P;
  g.block = NT;
  g.persistent = persist;
  std::ostringstream info;
  info << "gemm " << M << "x" << N << "x" << K << (rq.dtype == LEGO_BF16 ? " bf16" : " f16") << " tile " << bm << "x"
       << bn << "x" << bk << " waves " << NWM << "x" << NWN << " wave " << wm << "x" << wn << " mfma " << MB << "x"
       << MB << "x" << KB << " sched" << (xcd ? "+xcd" : "") << " A:V" << ops[0].V
       << (ops[0].gaxis == 2 ? "b" + std::to_string(ops[0].VR) + "x" + std::to_string(ops[0].VC) : (ops[0].gaxis ? "k" : "m"))
       << (ops[0].sep ? " sep" : " full") << (ops[0].svec ? " svec" : " sscalar")
       << (ops[0].frvec ? " frvec" : (ops[0].frtr ? " frtr" : (ops[0].frzp ? " frzpair" : (ops[0].frdw ? " frdw" : " frscalar")))) << " B:V" << ops[1].V
       << (ops[1].gaxis == 2 ? "b" + std::to_string(ops[1].VR) + "x" + std::to_string(ops[1].VC) : (ops[1].gaxis ? "k" : "n"))
       << (ops[1].sep ? " sep" : " full") << (ops[1].svec ? " svec" : " sscalar")
       << (ops[1].frvec ? " frvec" : (ops[1].frtr ? " frtr" : (ops[1].frdw ? " frdw" : " frscalar"))) << (csep ? " C:sep" : " C:full") << (wide ? " i64" : " u32")
       << (direct ? " direct-lds" : " staged")
       << (direct ? std::string(dma_spread ? " spread" : " burst") + " fd" + std::to_string(frag_dist) : "")
       << (ragged_groups ? " ragged-groups" : "")
       << (ops[0].edge || ops[1].edge || cedge ? " edges" : "") << (persist ? " persistent" : "") << " stages " << nstages << " lds " << nstages * stage_bytes
       << "B ops" << opsinfo.str();
  g.info = info.str();
  g.wide_ok = direct && !((ops[0].frtr || ops[1].frtr) && (ops[0].edge || ops[1].edge || cedge));
  return g;
}

}  // namespace

GemmPlan plan_gemm(const GemmRequest& rq) {
  // 128x128 wave tiles (4 waves) win where the copies are direct: 0.852
  // against 0.876 ms for 8 waves of 128x64 on the 8192^3 bf16 GEMM, reading
  // 1/3 less LDS per MFMA, and 1-5% with transposing fragment reads (8192^3
  // fp16 A row-major, B row-major: 1241-1248 -> 1264-1269 TFLOP/s; A column-
  // major: 1215-1219 -> 1244-1254).  Register-staged plans keep two waves per
  // SIMD (4096^3 Morton-A GEMM: 908-937 TFLOP/s with 8 waves, 833-872 with
  // 4), and so do plans with transposing reads and padded tiles (1000^3
  // fp16, A column-major: 176 VGPRs spilled with 4 waves).
  GemmPlan p = plan_gemm_waves(rq, true);
  const long long wide = tune("gemm.wide_waves", -1);  // -1: the rule above
  if (rq.wn || (wide < 0 ? p.wide_ok : wide != 0)) return p;
  return plan_gemm_waves(rq, false);
}

namespace {
std::mutex g_mu;
std::map<std::string, std::pair<std::vector<LayoutP>, std::shared_ptr<GemmPlan>>> g_cache;
}  // namespace

std::shared_ptr<GemmPlan> gemm_plan_cached(const GemmRequest& rq) {
  std::ostringstream k;
  k << rq.M << "," << rq.N << "," << rq.K << "," << rq.dtype << "," << rq.bm << "," << rq.bn << "," << rq.bk << ","
    << rq.wm << "," << rq.wn << "," << rq.group_m << "," << rq.xcd << "," << rq.stages;
  for (auto* l : {&rq.a, &rq.b, &rq.c, &rq.sched, &rq.lds_a, &rq.lds_b, &rq.frag_a, &rq.frag_b, &rq.frag_c})
    k << "," << (const void*)l->get();
  std::string key = k.str();
  {
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_cache.find(key);
    if (it != g_cache.end()) return it->second.second;
  }
  auto p = std::make_shared<GemmPlan>(plan_gemm(rq));
  std::lock_guard<std::mutex> lk(g_mu);
  g_cache[key] = {{rq.a, rq.b, rq.c, rq.sched, rq.lds_a, rq.lds_b, rq.frag_a, rq.frag_b, rq.frag_c}, p};
  return p;
}

std::vector<std::pair<std::string, std::string>> selftest_sources() {
  std::vector<std::pair<std::string, std::string>> out;
  // Index maps of the 128 x 128 three-level tiled layout.
  LayoutP c1 = make_tileorderby({make_row({2, 2}), make_row({4, 4}), make_row({16, 16})});
  out.push_back({"index apply 128x128 tiled", plan_index_eval(*c1, 0, 4).src});
  out.push_back({"index inv 128x128 tiled", plan_index_eval(*c1, 1, 4).src});
  // Row <-> blocked remap of 8192^2 fp32.
  LayoutP row = make_from_piece(make_row({8192, 8192}));
  LayoutP blk = make_tileorderby({make_col({128, 128}), make_row({64, 64})});
  out.push_back({"remap row->blocked f32", plan_remap(*row, *blk, 4).src});
  out.push_back({"remap blocked->row f32", plan_remap(*blk, *row, 4).src});
  // Row <-> Morton remap of 4096^2 fp16, and the transpose.
  LayoutP r4 = make_from_piece(make_row({4096, 4096}));
  LayoutP mz = make_from_piece(make_genp(GEN_MORTON, {4096, 4096}, {}));
  out.push_back({"remap row->morton f16", plan_remap(*r4, *mz, 2).src});
  out.push_back({"remap morton->row f16", plan_remap(*mz, *r4, 2).src});
  LayoutP col = make_from_piece(make_col({8192, 8192}));
  out.push_back({"remap row->col f32", plan_remap(*row, *col, 4).src});
  // Row <-> antidiagonal order of 4096^2 fp32 (the box path).
  LayoutP ad = make_from_piece(make_genp(GEN_ANTIDIAG, {4096, 4096}, {}));
  LayoutP r4f = make_from_piece(make_row({4096, 4096}));
  out.push_back({"remap row->antidiag f32", plan_remap(*r4f, *ad, 4).src});
  out.push_back({"remap antidiag->row f32", plan_remap(*ad, *r4f, 4).src});
  // GEMMs.
  GemmRequest g1;
  g1.M = g1.N = g1.K = 128;
  g1.dtype = LEGO_F16;
  g1.bm = g1.bn = 64;
  g1.bk = 32;
  g1.wm = g1.wn = 16;
  out.push_back({"gemm 128^3 f16 64x64x32 wave 16x16", plan_gemm(g1).src});
  GemmRequest g3;
  g3.M = g3.N = g3.K = 1024;
  g3.dtype = LEGO_F16;
  g3.bm = g3.bn = 128;
  g3.bk = 32;
  g3.wm = g3.wn = 64;
  out.push_back({"gemm 1024^3 f16 128x128x32", plan_gemm(g3).src});
  GemmRequest g4;
  g4.M = g4.N = g4.K = 8192;
  g4.dtype = LEGO_BF16;
  g4.xcd = 1;
  out.push_back({"gemm 8192^3 bf16 256x256x64", plan_gemm(g4).src});
  GemmRequest g5;
  g5.M = g5.N = g5.K = 4096;
  g5.dtype = LEGO_F16;
  g5.a = mz;
  g5.b = r4;
  g5.xcd = 1;
  out.push_back({"gemm 4096^3 f16 morton A, row B", plan_gemm(g5).src});
  // Operands contiguous along m or n: fragments through the transposing LDS
  // load (B row-major: B only; A column-major too: both).
  LayoutP c4 = make_from_piece(make_col({4096, 4096}));
  for (int both = 0; both < 2; ++both) {
    GemmRequest g6;
    g6.M = g6.N = g6.K = 4096;
    g6.dtype = LEGO_F16;
    g6.a = both ? c4 : r4;
    g6.b = r4;
    g6.xcd = 1;
    out.push_back({both ? "gemm 4096^3 f16 col A, row B" : "gemm 4096^3 f16 row A, row B", plan_gemm(g6).src});
  }
  // Transposing reads with padded tiles (1000 = 3 * 256 + 232).
  GemmRequest g7;
  g7.M = g7.N = g7.K = 1000;
  g7.dtype = LEGO_F16;
  g7.a = make_from_piece(make_col({1000, 1000}));
  g7.b = make_from_piece(make_row({1000, 1000}));
  g7.xcd = 1;
  out.push_back({"gemm 1000^3 f16 col A, row B, padded tiles", plan_gemm(g7).src});
  return out;
}

}  // namespace lego
