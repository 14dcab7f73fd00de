"""Host execution of the generated index code ("fake device").

Every generated kernel source of the built-in configurations is cut before its
kernel template; the lowered index functions are compiled with g++ and run on
the CPU exactly as the kernels call them.  The harness checks that every
address stays inside its buffer and that every map is a bijection, and it
simulates the data movement the kernel performs (index maps, remaps) so the
result can be compared element by element with the oracle.  This catches
lowering and planning bugs before any GPU launch.
"""
import os
import subprocess
import tempfile

import numpy as np
import pytest

from oracle import layout as OL
from oracle import remap as OR

MARK = "// ---- template ----"

HARNESS_COMMON = r"""
#define LEGO_FN static inline
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <vector>
#define FAIL(...) do { fprintf(stderr, __VA_ARGS__); fprintf(stderr, "\n"); exit(1); } while (0)
"""

HARNESS_INDEX = r"""
int main(int argc, char** argv) {
  FILE* f = fopen(argv[1], "wb");
#ifdef LEGO_HAVE_APPLY
  for (u64 x = 0; x < NPOINTS; ++x) { long long v = (long long)lego_map((IDX_T)x); fwrite(&v, 8, 1, f); }
#else
  for (u64 p = 0; p < NPOINTS; ++p) {
    IDX_T o[RANK]; lego_inv((IDX_T)p, o);
    for (int k = 0; k < RANK; ++k) { long long v = (long long)o[k]; fwrite(&v, 8, 1, f); }
  }
#endif
  fclose(f);
  return 0;
}
"""

HARNESS_REMAP = r"""
int main(int argc, char** argv) {
#ifdef LEGO_REMAP_DIRECT
  const u64 n = NVEC * (u64)V;
  {  // the workgroup -> chunk schedule is a bijection onto the chunks
    const u64 chunk = (u64)NT * UNROLL, nblk = (NVEC + chunk - 1) / chunk;
    std::vector<char> hit(nblk);
    for (u64 b = 0; b < nblk; ++b) {
      u64 c = (u64)blk((IDX_T)b);
      if (c >= nblk || hit[c]++) FAIL("blk is not a bijection");
    }
  }
  const u64 nsrc = NSRC;
  std::vector<long long> perm(n, -2);  // dst element -> src element (-1: zero fill)
  for (u64 t = 0; t < NVEC; ++t) {
#if MASKED
    if (!src_ok((IDX_T)t)) {
      for (int e = 0; e < V; ++e) perm[t * V + e] = -1;
      continue;
    }
#endif
    u64 s = (u64)src_vec((IDX_T)t);
    if ((s + 1) * V > nsrc) FAIL("src_vec(%llu) = %llu out of range", (unsigned long long)t, (unsigned long long)s);
    for (int e = 0; e < V; ++e) perm[t * V + e] = (long long)(s * V + e);
  }
#elif defined(LEGO_REMAP_BOX)
  // The box kernel's lines (emulated): position l of line p of a BX x BX box;
  // the per-side offsets from the generated functions, split or whole.
  const u64 n = (u64)EXT0 * EXT1, nsrc = n;
  const long long NW = NT / 64;
  if (NT % 64 || NT > 256) FAIL("NT is not whole waves");
  if ((unsigned long long)BX * (BX + BPAD) * sizeof(ELEM_T) > 160 * 1024) FAIL("box exceeds 160 KiB of LDS");
  if (NBR != (EXT0 + BX - 1) / BX || NBC != (EXT1 + BX - 1) / BX) FAIL("box grid does not cover the extents");
  // position l on line p: row p, column p, or antidiagonals p (l <= p) and
  // p + BX (l > p); r is the row, column or antidiagonal of the element
  auto pt = [&](int ord, long long p, long long l, long long* a, long long* b, long long* r) {
    if (ord == 0) { *a = p; *b = l; *r = p; }
    else if (ord == 1) { *a = l; *b = p; *r = p; }
    else { *a = l; *b = (p - l) & (BX - 1); *r = *a + *b; }
  };
  std::vector<long long> perm(n, -2);
  std::vector<long long> tile((u64)BX * (BX + BPAD));
  std::vector<char> bseen((u64)NBR * NBC);
  for (u64 bx = 0; bx < (u64)NBR * NBC; ++bx) {
    IDX_T bi, bj;
    bord((IDX_T)bx, &bi, &bj);
    if (bi >= NBR || bj >= NBC || bseen[(u64)bi * NBC + bj]++) FAIL("bord is not a bijection onto the boxes");
    const u64 i0 = (u64)bi * BX, j0 = (u64)bj * BX;
    std::fill(tile.begin(), tile.end(), -1);
    std::vector<char> rseen(BX * BX), wseen(BX * BX);
    for (long long it = 0; it * NW < BX; ++it)
      for (long long w = 0; w < NW; ++w)
        for (long long l = 0; l < BX; ++l) {  // position l of the line (lane l % 64)
          const long long p = it * NW + w;
          long long a, b, r;
          pt(S_ORD, p, l, &a, &b, &r);
          if (rseen[a * BX + b]++) FAIL("a box point is loaded twice");
          if (i0 + a >= (u64)EXT0 || j0 + b >= (u64)EXT1) continue;
#if S_SEP
          const u64 sa = (u64)(IDX_T)(s_u(bi, bj, (IDX_T)r) + s_l((IDX_T)l));
#else
          const u64 sa = (u64)s_f((IDX_T)(i0 + a), (IDX_T)(j0 + b));
#endif
          if (sa >= nsrc) FAIL("source offset out of range");
          tile[a * (BX + BPAD) + b] = (long long)sa;
        }
    for (long long it = 0; it * NW < BX; ++it)
      for (long long w = 0; w < NW; ++w)
        for (long long l = 0; l < BX; ++l) {  // position l of the line (lane l % 64)
          const long long p = it * NW + w;
          long long a, b, r;
          pt(D_ORD, p, l, &a, &b, &r);
          if (wseen[a * BX + b]++) FAIL("a box point is stored twice");
          if (i0 + a >= (u64)EXT0 || j0 + b >= (u64)EXT1) continue;
#if D_SEP
          const u64 d = (u64)(IDX_T)(d_u(bi, bj, (IDX_T)r) + d_l((IDX_T)l));
#else
          const u64 d = (u64)d_f((IDX_T)(i0 + a), (IDX_T)(j0 + b));
#endif
          if (d >= n) FAIL("destination offset out of range");
          if (perm[d] != -2) FAIL("destination written twice");
          if (tile[a * (BX + BPAD) + b] < 0) FAIL("LDS slot read before written");
          perm[d] = tile[a * (BX + BPAD) + b];
        }
    for (long long q = 0; q < BX * BX; ++q)
      if (!rseen[q] || !wseen[q]) FAIL("a box point is not covered by the lines");
  }
#else
  const u64 n = NELEM, nsrc = NELEM;
#if LDS_BLOCK
  if (NT < 1 || NT > 256 || (TILE / (VL * NX)) % NT || (TILE / VS) % NT) FAIL("NT does not divide the tile's blocks");
  if (VL * NX != VS * NY) FAIL("a block holds NX source and NY destination vectors");
#else
  if (NT < 1 || NT > 256 || (TILE / VL) % NT || (TILE / VS) % NT) FAIL("NT does not divide the tile's vectors");
#endif
  if ((unsigned long long)TILE * sizeof(ELEM_T) > 131072) FAIL("LDS tile exceeds 128 KiB");
  if ((unsigned long long)TILE * sizeof(ELEM_T) / NT > 512) FAIL("too many tile elements per thread");
  std::vector<long long> perm(n, -2);
  std::vector<long long> tile(TILE);
  std::vector<char> wseen(TILE);
  for (u64 g = 0; g < NTILES; ++g) {
    std::fill(tile.begin(), tile.end(), -1);
#if LDS_BLOCK
    for (u64 b = 0; b < TILE / (VL * NX); ++b) {
      long long blk[VL * NX];
      for (u64 x = 0; x < NX; ++x) {
        u64 s = (u64)src_off((IDX_T)g, (IDX_T)b, (IDX_T)x);
        if (s % VL || s + VL > n) FAIL("src_off(%llu,%llu,%llu) = %llu bad", (unsigned long long)g, (unsigned long long)b, (unsigned long long)x, (unsigned long long)s);
        for (int e = 0; e < VL; ++e) blk[x * VL + e] = (long long)(s + e);
      }
      std::vector<char> used(VL * NX);
      for (u64 y = 0; y < NY; ++y) {
        u64 l = (u64)ldsw((IDX_T)b, (IDX_T)y);
        if (l % VS || l + VS > TILE) FAIL("ldsw out of range or misaligned");
        for (int e = 0; e < VS; ++e) {
          const int k = blk_el((int)(y * VS + e));
          if (k < 0 || k >= VL * NX || used[k]++) FAIL("blk_el is not a permutation of the block");
          if (g == 0) { if (wseen[l + e]++) FAIL("ldsw not injective"); }
          tile[l + e] = blk[k];
        }
      }
    }
#else
    for (u64 q = 0; q < TILE / VL; ++q) {
      u64 s = (u64)src_off((IDX_T)g, (IDX_T)q);
      if (s % VL || s + VL > n) FAIL("src_off(%llu,%llu) = %llu bad", (unsigned long long)g, (unsigned long long)q, (unsigned long long)s);
      for (int e = 0; e < VL; ++e) {
        u64 l = (u64)ldsw((IDX_T)q, (IDX_T)e);
        if (l >= TILE) FAIL("ldsw out of range");
        if (g == 0) { if (wseen[l]++) FAIL("ldsw not injective"); }
        tile[l] = (long long)(s + e);
      }
    }
#endif
    for (u64 q = 0; q < TILE / VS; ++q) {
      u64 l = (u64)ldsr((IDX_T)q);
      u64 d = (u64)dst_off((IDX_T)g, (IDX_T)q);
      if (l % VS || l + VS > TILE) FAIL("ldsr out of range");
      if (d % VS || d + VS > n) FAIL("dst_off out of range");
      for (int e = 0; e < VS; ++e) {
        if (perm[d + e] != -2) FAIL("destination written twice");
        if (tile[l + e] < 0) FAIL("LDS slot read before written");
        perm[d + e] = tile[l + e];
      }
    }
  }
#endif
  std::vector<char> seen(nsrc);
  for (u64 i = 0; i < n; ++i) {
    if (perm[i] == -2) FAIL("destination %llu never written", (unsigned long long)i);
    if (perm[i] >= 0 && seen[perm[i]]++) FAIL("source read twice");
  }
  FILE* f = fopen(argv[1], "wb");
  fwrite(perm.data(), 8, n, f);
  fclose(f);
  return 0;
}
"""

# Bounds and bijectivity of a remap too large to simulate element by element:
# one bit per destination element written and per source element read.
HARNESS_REMAP_BITS = r"""
struct Bits {
  std::vector<unsigned long long> w;
  explicit Bits(u64 n) : w((n + 63) / 64) {}
  bool set(u64 i) { unsigned long long m = 1ull << (i % 64), o = w[i / 64]; w[i / 64] = o | m; return o & m; }
  bool all(u64 n) const { for (u64 i = 0; i < n; ++i) if (!(w[i / 64] >> (i % 64) & 1)) return false; return true; }
};
int main() {
  // vectors are aligned runs, so one bit per source / destination vector
#ifdef LEGO_REMAP_DIRECT
  {  // the workgroup -> chunk schedule is a bijection onto the chunks
    const u64 chunk = (u64)NT * UNROLL, nblk = (NVEC + chunk - 1) / chunk;
    Bits hit(nblk);
    for (u64 b = 0; b < nblk; ++b) {
      u64 c = (u64)blk((IDX_T)b);
      if (c >= nblk || hit.set(c)) FAIL("blk is not a bijection");
    }
  }
  Bits rd(NSRC / V), wr(NVEC);
  for (u64 t = 0; t < NVEC; ++t) {
    u64 s = (u64)src_vec((IDX_T)t);
    if ((s + 1) * V > NSRC) FAIL("src_vec out of range");
    if (rd.set(s)) FAIL("source read twice");
    wr.set(t);
  }
  if (!rd.all(NSRC / V) || !wr.all(NVEC)) FAIL("element never copied");
#else
  const u64 n = NELEM;
#if LDS_BLOCK
  if (NT < 1 || NT > 256 || (TILE / (VL * NX)) % NT || (TILE / VS) % NT) FAIL("NT does not divide the tile's blocks");
  if (VL * NX != VS * NY) FAIL("a block holds NX source and NY destination vectors");
#else
  if (NT < 1 || NT > 256 || (TILE / VL) % NT || (TILE / VS) % NT) FAIL("NT does not divide the tile's vectors");
#endif
  Bits rd(n / VL), wr(n / VS);
  for (u64 g = 0; g < NTILES; ++g) {
#if LDS_BLOCK
    for (u64 b = 0; b < TILE / (VL * NX); ++b)
      for (u64 x = 0; x < NX; ++x) {
        u64 s = (u64)src_off((IDX_T)g, (IDX_T)b, (IDX_T)x);
        if (s % VL || s + VL > n) FAIL("src_off out of range");
        if (rd.set(s / VL)) FAIL("source read twice");
      }
#else
    for (u64 q = 0; q < TILE / VL; ++q) {
      u64 s = (u64)src_off((IDX_T)g, (IDX_T)q);
      if (s % VL || s + VL > n) FAIL("src_off out of range");
      if (rd.set(s / VL)) FAIL("source read twice");
    }
#endif
    for (u64 q = 0; q < TILE / VS; ++q) {
      u64 d = (u64)dst_off((IDX_T)g, (IDX_T)q);
      if (d % VS || d + VS > n) FAIL("dst_off out of range");
      if (wr.set(d / VS)) FAIL("destination written twice");
    }
  }
  if (!rd.all(n / VL) || !wr.all(n / VS)) FAIL("element never copied");
#endif
  printf("ok\n");
  return 0;
}
"""

HARNESS_GEMM = r"""
static u64 goff_a(u64 tm, u64 kt, u64 tid, u64 u) {
#if A_SEP
  return (u64)a_gt((IDX_T)tm) + (u64)a_gk((IDX_T)kt) + (u64)a_gl((IDX_T)tid, (IDX_T)u);
#else
  return (u64)a_gf((IDX_T)tm, (IDX_T)kt, (IDX_T)tid, (IDX_T)u);
#endif
}
static u64 goff_b(u64 tn, u64 kt, u64 tid, u64 u) {
#if B_SEP
  return (u64)b_gt((IDX_T)tn) + (u64)b_gk((IDX_T)kt) + (u64)b_gl((IDX_T)tid, (IDX_T)u);
#else
  return (u64)b_gf((IDX_T)tn, (IDX_T)kt, (IDX_T)tid, (IDX_T)u);
#endif
}
int main() {
  // schedule: a bijection of workgroups onto tiles
  std::vector<char> seen(GEMM_MT * GEMM_NT);
  for (u64 pid = 0; pid < GEMM_MT * GEMM_NT; ++pid) {
    IDX_T tm, tn; sched((IDX_T)pid, &tm, &tn);
    if ((u64)tm >= GEMM_MT || (u64)tn >= GEMM_NT) FAIL("sched out of range");
    if (seen[(u64)tm * GEMM_NT + tn]++) FAIL("sched not injective");
  }
  // global loads: every element of A (B) loaded exactly once per tile row (column)
  {
    std::vector<char> a(GEMM_M * GEMM_K);
    for (u64 tm = 0; tm < GEMM_MT; ++tm) for (u64 kt = 0; kt < KT; ++kt)
      for (u64 tid = 0; tid < NT; ++tid) for (u64 u = 0; u < A_NV; ++u) {
        if (A_GUARD && u * NT + tid >= A_NVEC) continue;
#if A_EDGE
        if (!a_ok((IDX_T)tm, (IDX_T)kt, (IDX_T)tid, (IDX_T)u)) continue;  // padding, read as zero
#endif
        u64 o = goff_a(tm, kt, tid, u);
        if (o % A_V || o + A_V > GEMM_M * GEMM_K) FAIL("A offset out of range");
        for (int e = 0; e < A_V; ++e) if (a[o + e]++) FAIL("A element loaded twice");
      }
    for (char c : a) if (c != 1) FAIL("A element never loaded");
  }
  {
    std::vector<char> b(GEMM_K * GEMM_N);
    for (u64 tn = 0; tn < GEMM_NT; ++tn) for (u64 kt = 0; kt < KT; ++kt)
      for (u64 tid = 0; tid < NT; ++tid) for (u64 u = 0; u < B_NV; ++u) {
        if (B_GUARD && u * NT + tid >= B_NVEC) continue;
#if B_EDGE
        if (!b_ok((IDX_T)tn, (IDX_T)kt, (IDX_T)tid, (IDX_T)u)) continue;
#endif
        u64 o = goff_b(tn, kt, tid, u);
        if (o % B_V || o + B_V > GEMM_K * GEMM_N) FAIL("B offset out of range");
        for (int e = 0; e < B_V; ++e) if (b[o + e]++) FAIL("B element loaded twice");
      }
    for (char c : b) if (c != 1) FAIL("B element never loaded");
  }
#if DIRECT_LDS
  // direct copies: load vector q of a thread lands in LDS slot q, which the
  // LDS layout must assign to exactly the elements that vector carries
  for (u64 tid = 0; tid < NT; ++tid) {
    for (u64 u = 0; u < A_NV; ++u) for (int e = 0; e < 8; ++e)
      if ((u64)a_s((IDX_T)tid, (IDX_T)u, (IDX_T)e) != (u * NT + tid) * 8 + e) FAIL("direct A slot mismatch");
    for (u64 u = 0; u < B_NV; ++u) for (int e = 0; e < 8; ++e)
      if ((u64)b_s((IDX_T)tid, (IDX_T)u, (IDX_T)e) != (u * NT + tid) * 8 + e) FAIL("direct B slot mismatch");
  }
  if ((unsigned long long)NSTAGES * (BM + BN) * BK * 2 > 160 * 1024) FAIL("LDS ring exceeds 160 KiB");
#endif
  // LDS stores: a bijection onto each stage
  {
    std::vector<char> la(BM * BK), lb(BN * BK);
    for (u64 tid = 0; tid < NT; ++tid) {
      for (u64 u = 0; u < A_NV; ++u) {
        if (A_GUARD && u * NT + tid >= A_NVEC) continue;
        for (int e = 0; e < A_V; ++e) { u64 o = a_s((IDX_T)tid, (IDX_T)u, (IDX_T)e); if (o >= BM * BK || la[o]++) FAIL("a_s bad"); }
      }
      for (u64 u = 0; u < B_NV; ++u) {
        if (B_GUARD && u * NT + tid >= B_NVEC) continue;
        for (int e = 0; e < B_V; ++e) { u64 o = b_s((IDX_T)tid, (IDX_T)u, (IDX_T)e); if (o >= BN * BK || lb[o]++) FAIL("b_s bad"); }
      }
    }
    for (char c : la) if (c != 1) FAIL("LDS A slot never written");
    for (char c : lb) if (c != 1) FAIL("LDS B slot never written");
  }
  // fragment reads stay inside the stage; each wave reads its rows x all k
  for (u64 w = 0; w < NWAVES; ++w) {
    std::vector<int> ra(BM * BK), rb(BN * BK);
    for (u64 lane = 0; lane < 64; ++lane) for (u64 s = 0; s < BK / KB; ++s) for (int e = 0; e < 8; ++e) {
      for (u64 mi = 0; mi < MI; ++mi) { u64 o = a_fr((IDX_T)lane, (IDX_T)w, (IDX_T)mi, (IDX_T)s, (IDX_T)e); if (o >= BM * BK) FAIL("a_fr out of range"); ra[o]++; }
      for (u64 ni = 0; ni < NI; ++ni) { u64 o = b_fr((IDX_T)lane, (IDX_T)w, (IDX_T)ni, (IDX_T)s, (IDX_T)e); if (o >= BN * BK) FAIL("b_fr out of range"); rb[o]++; }
    }
    long long na = 0, nb = 0;
    for (int c : ra) { if (c > 1) FAIL("a_fr duplicates"); na += c != 0; }
    for (int c : rb) if (c > 1) FAIL("b_fr duplicates");
    for (int c : rb) nb += c != 0;
    if (na != (long long)MI * MB * BK || nb != (long long)NI * MB * BK) FAIL("fragments do not cover the wave tile");
  }
  // transposing fragment reads: lane i of 16-lane block b receives element j
  // of half h from the address of lane 16b + 4j + i/4, plus i%4; that must be
  // the element the fragment layout gives (lane, 4h + j)
#if A_FRTR || B_FRTR
  for (u64 w = 0; w < NWAVES; ++w)
    for (u64 s = 0; s < BK / KB; ++s) for (u64 h = 0; h < 2; ++h) for (u64 l = 0; l < 64; ++l) for (u64 j = 0; j < 4; ++j) {
      u64 sup = 16 * (l / 16) + 4 * j + (l % 16) / 4;
#if A_FRTR
      for (u64 mi = 0; mi < MI; ++mi) {
        u64 o = a_ft((IDX_T)sup, (IDX_T)w, (IDX_T)mi, (IDX_T)s, (IDX_T)h);
        if (o % 4 || o + 4 > BM * BK) FAIL("a_ft misaligned or out of range");
        if (o + l % 4 != (u64)a_fr((IDX_T)l, (IDX_T)w, (IDX_T)mi, (IDX_T)s, (IDX_T)(4 * h + j))) FAIL("a_ft mismatch");
      }
#endif
#if B_FRTR
      for (u64 ni = 0; ni < NI; ++ni) {
        u64 o = b_ft((IDX_T)sup, (IDX_T)w, (IDX_T)ni, (IDX_T)s, (IDX_T)h);
        if (o % 4 || o + 4 > BN * BK) FAIL("b_ft misaligned or out of range");
        if (o + l % 4 != (u64)b_fr((IDX_T)l, (IDX_T)w, (IDX_T)ni, (IDX_T)s, (IDX_T)(4 * h + j))) FAIL("b_ft mismatch");
      }
#endif
    }
#endif
  // dword fragment reads: elements 2p, 2p + 1 adjacent and 4-byte aligned;
  // with a constant distance D, dword 2h at a_fd(h) and dword 2h + 1 at +D
#if A_FRDW || B_FRDW
  for (u64 w = 0; w < NWAVES; ++w)
    for (u64 s = 0; s < BK / KB; ++s) for (u64 l = 0; l < 64; ++l) for (u64 p = 0; p < 4; ++p) {
#if A_FRDW
      for (u64 mi = 0; mi < MI; ++mi) {
        u64 o = a_fr((IDX_T)l, (IDX_T)w, (IDX_T)mi, (IDX_T)s, (IDX_T)(2 * p));
        if (o % 2 || (u64)a_fr((IDX_T)l, (IDX_T)w, (IDX_T)mi, (IDX_T)s, (IDX_T)(2 * p + 1)) != o + 1) FAIL("a_fr dword pair");
#if A_FRDW_D
        if ((u64)a_fd((IDX_T)l, (IDX_T)w, (IDX_T)mi, (IDX_T)s, (IDX_T)(p / 2)) + (p % 2) * A_FRDW_D != o) FAIL("a_fd mismatch");
#endif
      }
#endif
#if B_FRDW
      for (u64 ni = 0; ni < NI; ++ni) {
        u64 o = b_fr((IDX_T)l, (IDX_T)w, (IDX_T)ni, (IDX_T)s, (IDX_T)(2 * p));
        if (o % 2 || (u64)b_fr((IDX_T)l, (IDX_T)w, (IDX_T)ni, (IDX_T)s, (IDX_T)(2 * p + 1)) != o + 1) FAIL("b_fr dword pair");
#if B_FRDW_D
        if ((u64)b_fd((IDX_T)l, (IDX_T)w, (IDX_T)ni, (IDX_T)s, (IDX_T)(p / 2)) + (p % 2) * B_FRDW_D != o) FAIL("b_fd mismatch");
#endif
      }
#endif
    }
#endif
  // row-pair fragment reads: element 4h + 2t + q of block 2m + p at
  // a_fz(m, h) + 4t + 2p + q, a_fz a multiple of 8
#if A_FRZP
  for (u64 w = 0; w < NWAVES; ++w)
    for (u64 s = 0; s < BK / KB; ++s) for (u64 l = 0; l < 64; ++l) for (u64 m = 0; m < MI / 2; ++m)
      for (u64 h = 0; h < 2; ++h) {
        u64 z = a_fz((IDX_T)l, (IDX_T)w, (IDX_T)m, (IDX_T)s, (IDX_T)h);
        if (z % 8 || z + 8 > BM * BK) FAIL("a_fz misaligned or out of range");
        for (u64 p = 0; p < 2; ++p) for (u64 t = 0; t < 2; ++t) for (u64 q = 0; q < 2; ++q)
          if ((u64)a_fr((IDX_T)l, (IDX_T)w, (IDX_T)(2 * m + p), (IDX_T)s, (IDX_T)(4 * h + 2 * t + q)) != z + 4 * t + 2 * p + q)
            FAIL("a_fz mismatch");
      }
#endif
  // epilogue: every C element written exactly once
  {
    std::vector<char> c(GEMM_M * GEMM_N);
    for (u64 tm = 0; tm < GEMM_MT; ++tm) for (u64 tn = 0; tn < GEMM_NT; ++tn)
      for (u64 lane = 0; lane < 64; ++lane) for (u64 w = 0; w < NWAVES; ++w)
        for (u64 mi = 0; mi < MI; ++mi) for (u64 ni = 0; ni < NI; ++ni) for (u64 r = 0; r < (MB == 32 ? 16 : 4); ++r) {
#if C_EDGE
          if (!c_ok((IDX_T)tm, (IDX_T)tn, (IDX_T)lane, (IDX_T)w, (IDX_T)mi, (IDX_T)ni, (IDX_T)r)) continue;
#endif
#if C_SEP
          u64 o = (u64)c_t((IDX_T)tm, (IDX_T)tn) + (u64)c_l((IDX_T)lane, (IDX_T)w, (IDX_T)mi, (IDX_T)ni, (IDX_T)r);
#else
          u64 o = (u64)c_f((IDX_T)tm, (IDX_T)tn, (IDX_T)lane, (IDX_T)w, (IDX_T)mi, (IDX_T)ni, (IDX_T)r);
#endif
          if (o >= GEMM_M * GEMM_N || c[o]++) FAIL("C offset bad");

        }
  }
  printf("ok\n");
  return 0;
}
"""


def _sources():
    import paper_2505_08091_amd as L
    return L.selftest_sources()


def _oracle_for(name):
    """Oracle layouts (and element size) behind each built-in generated source."""
    c1 = OL.TileOrderBy(OL.Row(2, 2), OL.Row(4, 4), OL.Row(16, 16))
    row8 = OL.as_layout(OL.Row(8192, 8192))
    blk = OL.TileOrderBy(OL.Col(128, 128), OL.Row(64, 64))
    r4 = OL.as_layout(OL.Row(4096, 4096))
    mz = OL.as_layout(OL.morton_genp(4096, 4096))
    return {
        "index apply 128x128 tiled": ("apply", c1),
        "index inv 128x128 tiled": ("inv", c1),
        "remap row->blocked f32": ("remap", row8, blk),
        "remap blocked->row f32": ("remap", blk, row8),
        "remap row->morton f16": ("remap", r4, mz),
        "remap morton->row f16": ("remap", mz, r4),
        "remap row->col f32": ("remap", row8, OL.as_layout(OL.Col(8192, 8192))),
        "remap row->antidiag f32": ("remap", OL.as_layout(OL.Row(4096, 4096)), OL.as_layout(OL.antidiag_genp(4096))),
        "remap antidiag->row f32": ("remap", OL.as_layout(OL.antidiag_genp(4096)), OL.as_layout(OL.Row(4096, 4096))),
    }.get(name)


def _compile_and_run(src, harness, tmp, args=()):
    head = src.split(MARK)[0]
    cpp = os.path.join(tmp, "h.cpp")
    exe = os.path.join(tmp, "h")
    with open(cpp, "w") as f:
        f.write(HARNESS_COMMON + head + harness)
    r = subprocess.run(["g++", "-O2", "-std=c++17", "-w", cpp, "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    r = subprocess.run([exe, *args], capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    return r.stdout


N_SOURCES = 16


def test_source_count():
    assert len(_sources()) == N_SOURCES


@pytest.mark.parametrize("i", range(N_SOURCES))
def test_generated_source_on_host(i):
    name, src = _sources()[i]
    assert MARK in src
    with tempfile.TemporaryDirectory() as tmp:
        out = os.path.join(tmp, "out.bin")
        if "LEGO_HAVE_APPLY" in src or "LEGO_HAVE_INV" in src:
            kind, lay = _oracle_for(name)
            _compile_and_run(src, HARNESS_INDEX, tmp, [out])
            got = np.fromfile(out, dtype=np.int64)
            if kind == "apply":
                assert (got == OL.apply_all(lay)).all(), name
            else:
                assert (got.reshape(-1, 2) == OL.inv_all(lay)).all(), name
        elif "LEGO_REMAP_" in src:
            kind, ls, ld = _oracle_for(name)
            _compile_and_run(src, HARNESS_REMAP, tmp, [out])
            perm = np.fromfile(out, dtype=np.int64)
            # the oracle moves element indices: dst[L_dst(x)] = src[L_src(x)]
            exp = OR.remap(ls, ld, np.arange(ls.size(), dtype=np.int64))
            assert (perm == exp).all(), name
        else:
            assert "lego_gemm" in src
            assert _compile_and_run(src, HARNESS_GEMM, tmp).strip() == "ok", name


# ------------------------------------------------------------------------
# Every configuration the GPU tests launch, checked on the host first.
def _index_cases():
    import paper_2505_08091_amd as L
    from tests.test_gpu_genexpr import _wavefront
    from tests.test_gpu_index import _cases
    return _cases(L) + [("wavefront 1024^2 of 32x32 tiles", _wavefront(L, None, 1024, 32), _wavefront(None, OL, 1024, 32))]


def test_index_sources_of_gpu_cases():
    import paper_2505_08091_amd as L
    with tempfile.TemporaryDirectory() as tmp:
        out = os.path.join(tmp, "out.bin")
        for name, lay, olay in _index_cases():
            for kind in ("apply", "inv"):
                src = L.plan_source(kind, lay, param=8)
                _compile_and_run(src, HARNESS_INDEX, tmp, [out])
                got = np.fromfile(out, dtype=np.int64)
                if kind == "apply":
                    assert (got == OL.apply_all(olay)).all(), name
                else:
                    assert (got.reshape(-1, len(olay.dims())) == OL.inv_all(olay)).all(), name


@pytest.mark.parametrize("i", range(20))
def test_remap_sources_of_random_expand_and_box_cases(i):
    """The seeded random ExpandBy and antidiagonal remaps of the GPU tests,
    both directions, on the host (padding reads -1 here: zero fill)."""
    import paper_2505_08091_amd as L
    from tests.test_gpu_remap import _random_box_cases, _random_expand_cases
    name, ls, ld, ols, old, elem = (_random_expand_cases(L) + _random_box_cases(L))[i]
    with tempfile.TemporaryDirectory() as tmp:
        out = os.path.join(tmp, "out.bin")
        for a, b, oa, ob in ((ls, ld, ols, old), (ld, ls, old, ols)):
            src = L.plan_source("remap", a, b, param=elem)
            _compile_and_run(src, HARNESS_REMAP, tmp, [out])
            perm = np.fromfile(out, dtype=np.int64)
            exp = OR.remap(oa, ob, np.arange(1, OR.phys_size(oa) + 1, dtype=np.int64)) - 1
            assert (perm == exp).all(), name


def test_index_sources_of_random_cases():
    import paper_2505_08091_amd as L
    from tests.test_gpu_index import _random_index_cases
    with tempfile.TemporaryDirectory() as tmp:
        out = os.path.join(tmp, "out.bin")
        for name, lay, olay in _random_index_cases(L):
            for kind in ("apply", "inv"):
                src = L.plan_source(kind, lay, param=8)
                _compile_and_run(src, HARNESS_INDEX, tmp, [out])
                got = np.fromfile(out, dtype=np.int64)
                if kind == "apply":
                    assert (got == OL.apply_all(olay)).all(), name
                else:
                    assert (got.reshape(-1, len(olay.dims())) == OL.inv_all(olay)).all(), name


def _remap_cases():
    import paper_2505_08091_amd as L
    from tests.test_gpu_genexpr import _expr_cases
    from tests.test_gpu_remap import _expand_cases, _small_cases
    cases = [(n, ls, ld, ols, old) for n, ls, ld, ols, old in _small_cases(L) + _expand_cases(L) + _expr_cases(L)]
    for n in (2048, 4096, 8192, 1024):
        cases.append((f"transpose {n}", L.as_layout(L.Row(n, n)), L.as_layout(L.Col(n, n)),
                      OL.as_layout(OL.Row(n, n)), OL.as_layout(OL.Col(n, n))))
    cases.append(("identity 8192", L.as_layout(L.Row(8192, 8192)), L.as_layout(L.Row(8192, 8192)),
                  OL.as_layout(OL.Row(8192, 8192)), OL.as_layout(OL.Row(8192, 8192))))
    from tests.test_gpu_genexpr import _wavefront
    cases.append(("wavefront 8192", L.as_layout(L.Row(8192, 8192)), _wavefront(L, None, 8192, 64),
                  OL.as_layout(OL.Row(8192, 8192)), _wavefront(None, OL, 8192, 64)))
    n, ne = 8000, 8192
    cases.append(("pad 8000 into 8192 blocked", L.ExpandBy([n, n], [ne, ne], L.as_layout(L.Row(ne, ne))),
                  L.TileOrderBy(L.Col(ne // 64, ne // 64), L.Row(64, 64)),
                  OL.ExpandBy([n, n], [ne, ne], OL.as_layout(OL.Row(ne, ne))),
                  OL.TileOrderBy(OL.Col(ne // 64, ne // 64), OL.Row(64, 64))))
    return cases


def _check_remap_sources(L, ls, ld, ols, old, elem_bytes, tmp, name):
    out = os.path.join(tmp, "out.bin")
    for a, b, oa, ob in ((ls, ld, ols, old), (ld, ls, old, ols)):
        src = L.plan_source("remap", a, b, param=elem_bytes)
        _compile_and_run(src, HARNESS_REMAP, tmp, [out])
        perm = np.fromfile(out, dtype=np.int64)
        # source element k is tagged k + 1, so zero fill reads as -1
        exp = OR.remap(oa, ob, np.arange(1, OR.phys_size(oa) + 1, dtype=np.int64)) - 1
        assert (perm == exp).all(), (name, elem_bytes)


_BIG = 1 << 23  # cases above this many elements run once each (4-byte elements), in parallel


@pytest.mark.parametrize("i", range(5))
def test_remap_sources_of_big_gpu_cases(i):
    import paper_2505_08091_amd as L
    big = [c for c in _remap_cases() if OL.prod(c[3].dims()) > _BIG]
    assert len(big) == 5
    name, ls, ld, ols, old = big[i]
    with tempfile.TemporaryDirectory() as tmp:
        _check_remap_sources(L, ls, ld, ols, old, 4, tmp, name)


@pytest.mark.parametrize("elem_bytes", [1, 2, 4, 8])
def test_remap_sources_of_gpu_cases(elem_bytes):
    import paper_2505_08091_amd as L
    with tempfile.TemporaryDirectory() as tmp:
        out = os.path.join(tmp, "out.bin")
        for name, ls, ld, ols, old in _remap_cases():
            if OL.prod(ols.dims()) > _BIG:
                continue
            for a, b, oa, ob in ((ls, ld, ols, old), (ld, ls, old, ols)):
                src = L.plan_source("remap", a, b, param=elem_bytes)
                _compile_and_run(src, HARNESS_REMAP, tmp, [out])
                perm = np.fromfile(out, dtype=np.int64)
                # source element k is tagged k + 1, so zero fill reads as -1
                exp = OR.remap(oa, ob, np.arange(1, OR.phys_size(oa) + 1, dtype=np.int64)) - 1
                assert (perm == exp).all(), (name, elem_bytes)


@pytest.mark.parametrize("i", range(24))
def test_remap_sources_of_random_cases(i):
    """The seeded random remaps of the GPU tests, both directions, on the host."""
    import paper_2505_08091_amd as L
    from tests.test_gpu_remap import _random_remap_cases
    name, ls, ld, ols, old, elem = _random_remap_cases(L)[i]
    with tempfile.TemporaryDirectory() as tmp:
        out = os.path.join(tmp, "out.bin")
        for a, b, oa, ob in ((ls, ld, ols, old), (ld, ls, old, ols)):
            src = L.plan_source("remap", a, b, param=elem)
            _compile_and_run(src, HARNESS_REMAP, tmp, [out])
            perm = np.fromfile(out, dtype=np.int64)
            exp = OR.remap(oa, ob, np.arange(1, OR.phys_size(oa) + 1, dtype=np.int64)) - 1
            assert (perm == exp).all(), name


def _huge_remap_cases():
    """Remaps of 65600^2 one-byte elements (more than 2^32, so byte and element
    offsets need 64 bits; 65600 = 64 * 1025 has odd factors)."""
    import paper_2505_08091_amd as L
    n = 65600
    row = L.as_layout(L.Row(n, n))
    return [("row -> 64x64 blocked", row, L.TileOrderBy(L.Col(n // 64, n // 64), L.Row(64, 64))),
            ("row -> col", row, L.as_layout(L.Col(n, n)))]


@pytest.mark.slow
def test_remap_sources_beyond_4g_elements():
    import paper_2505_08091_amd as L
    with tempfile.TemporaryDirectory() as tmp:
        for name, ls, ld in _huge_remap_cases():
            for a, b in ((ls, ld), (ld, ls)):
                src = L.plan_source("remap", a, b, param=1)
                assert _compile_and_run(src, HARNESS_REMAP_BITS, tmp).strip() == "ok", name


def _gemm_cases():
    import paper_2505_08091_amd as L
    cases = []
    for dt in ("f16", "bf16"):
        cases.append(dict(M=128, N=128, K=128, dtype=dt, bm=64, bn=64, bk=32, wm=16, wn=16))
    cases.append(dict(M=1024, N=1024, K=1024, dtype="f16", bm=128, bn=128, bk=32, wm=64, wn=64, group_m=8))
    cases.append(dict(M=512, N=768, K=1024, dtype="bf16"))
    for la in ("Row", "Col"):
        for lb in ("Row", "Col"):
            cases.append(dict(M=256, N=512, K=384, dtype="f16", a=L.as_layout(getattr(L, la)(256, 384)),
                              b=L.as_layout(getattr(L, lb)(384, 512)), c=L.as_layout(L.Col(256, 512)),
                              bm=128, bn=128, bk=64, wm=64, wn=64))
    cases.append(dict(M=64, N=64, K=64, dtype="f16", bm=64, bn=64, bk=32, wm=32, wn=32))
    cases.append(dict(M=64, N=64, K=64, dtype="f16", bm=64, bn=64, bk=32, wm=16, wn=16))
    cases.append(dict(M=8192, N=8192, K=8192, dtype="bf16"))
    cases.append(dict(M=4096, N=4096, K=4096, dtype="f16", a=L.as_layout(L.GenP("morton", [4096, 4096])),
                      b=L.as_layout(L.Row(4096, 4096))))
    cases.append(dict(M=256, N=256, K=256, dtype="f16", bm=128, bn=128, bk=32, wm=64, wn=64))  # smoke
    for la, lb in (("Row", "Row"), ("Col", "Row"), ("Col", "Col")):  # m/n-contiguous operands, default plan
        cases.append(dict(M=2048, N=2048, K=2048, dtype="f16", a=L.as_layout(getattr(L, la)(2048, 2048)),
                          b=L.as_layout(getattr(L, lb)(2048, 2048))))
    for la in ("Row", "Col"):  # the four operand variants at 4096^3, default plan
        for lb in ("Row", "Col"):
            cases.append(dict(M=4096, N=4096, K=4096, dtype="f16", a=L.as_layout(getattr(L, la)(4096, 4096)),
                              b=L.as_layout(getattr(L, lb)(4096, 4096))))
    from tests.test_gpu_gemm import _ragged_cases
    cases += [{k: v for k, v in c.items() if k not in ("oa", "ob")} for c in _ragged_cases(L)]
    from tests.test_gpu_gemm import _sched_cases
    for _, sched, xcd in _sched_cases(L, 8, 8):
        cases.append(dict(M=2048, N=2048, K=512, dtype="bf16", sched=sched, xcd_remap=xcd))
    from tests import genp_exprs as GE
    sw = L.as_layout(L.GenPExpr([256, 64], GE.SWIZZLE64_APPLY, GE.SWIZZLE64_INV))
    cases.append(dict(M=1024, N=1024, K=1024, dtype="bf16", lds_a=sw, lds_b=sw))
    from tests.test_gpu_gemm import _persistent_cases
    cases += [{k: v for k, v in c.items() if k not in ("oa", "ob", "max_workgroups")} for c in _persistent_cases(L)]
    from tests.test_gpu_gemm import _morton_direct_cases, _morton_direct_kw
    cases += [{k: v for k, v in _morton_direct_kw(L, c).items() if k != "max_workgroups"} for c in _morton_direct_cases(L)]
    from tests.test_gpu_gemm import _random_cases
    cases += [{k: v for k, v in c.items() if k not in ("oa", "ob", "max_workgroups")} for c in _random_cases(L)]
    M, N, K = 32768, 256, 32768  # a 2 GiB operand
    cases.append(dict(M=M, N=N, K=K, dtype="bf16", a=L.as_layout(L.Row(M, K)), b=L.as_layout(L.Col(K, N))))
    cases.append(dict(M=M, N=N, K=K, dtype="bf16", a=L.as_layout(L.Col(M, K)), b=L.as_layout(L.Row(K, N))))
    return cases


N_GEMM_CASES = 86


def test_gemm_case_count():
    assert len(_gemm_cases()) == N_GEMM_CASES


@pytest.mark.parametrize("i", range(N_GEMM_CASES))
def test_gemm_sources_of_gpu_cases(i):
    import paper_2505_08091_amd as L
    kw = _gemm_cases()[i]
    src = L.plan_source("gemm", **kw)
    with tempfile.TemporaryDirectory() as tmp:
        assert _compile_and_run(src, HARNESS_GEMM, tmp).strip() == "ok", kw


HARNESS_ISQRT32_ALL = r"""
#include <omp.h>
int main() {
  // every 32-bit operand: r = floor(sqrt(v)) exactly
  unsigned long long bad = 0;
#pragma omp parallel for reduction(+ : bad) schedule(static)
  for (long long hi = 0; hi < 65536; ++hi)
    for (u64 lo = 0; lo < 65536; ++lo) {
      const u64 v = ((u64)hi << 16) | lo;
      const u64 r = lego_isqrt((u32)v);
      bad += !(r * r <= v && (r + 1) * (r + 1) > v);
    }
  printf("%llu\n", bad);
  return bad != 0;
}
"""


@pytest.mark.parametrize("estimate", ["float", "perturbed"])
def test_integer_square_root_32bit_exhaustive(estimate):
    """The 32-bit integer square root of the generated code on all 2^32
    operands.  It starts from a float square-root estimate and corrects it by
    integer comparisons; the second case replaces the estimate by one that is
    off by -2..+1 (a pseudo-random offset per operand), so exactness does not
    rest on how the device rounds its square root."""
    import paper_2505_08091_amd as L
    src = L.plan_source("apply", L.as_layout(L.GenP("antidiag", [64, 64])), param=4)
    head = src.split(MARK)[0]
    if estimate == "perturbed":
        head = ("static inline float lego_bad_sqrt(float x) {\n"
                "  const unsigned v = (unsigned)x;\n"
                "  const float s = __builtin_sqrtf(x) + (float)((int)((v * 2654435761u) >> 30) - 2);\n"
                "  return s < 0.f ? 0.f : s;\n"
                "}\n#define __builtin_sqrtf(x) lego_bad_sqrt(x)\n") + head
    with tempfile.TemporaryDirectory() as tmp:
        cpp, exe = os.path.join(tmp, "s.cpp"), os.path.join(tmp, "s")
        with open(cpp, "w") as f:
            f.write(HARNESS_COMMON + head + HARNESS_ISQRT32_ALL)
        r = subprocess.run(["g++", "-O2", "-std=c++17", "-fopenmp", "-w", cpp, "-o", exe], capture_output=True,
                           text=True)
        assert r.returncode == 0, r.stderr[-4000:]
        r = subprocess.run([exe], capture_output=True, text=True, timeout=600)
        assert r.returncode == 0 and r.stdout.strip() == "0", (r.stdout, r.stderr)


HARNESS_ISQRT = r"""
int main() {
  // 32-bit: every v below 2^20, and k^2 - 1, k^2, k^2 + 1 for every k < 2^16
  // (where a float estimate could round across the boundary), and the top.
  unsigned long long bad = 0;
  auto ok32 = [&](u64 v) {
    const u64 r = lego_isqrt((u32)v);
    if (!(r * r <= v && (r + 1) * (r + 1) > v)) ++bad;
  };
  for (u64 v = 0; v < (1ull << 20); ++v) ok32(v);
  for (u64 k = 1; k < (1ull << 16); ++k) { ok32(k * k - 1); ok32(k * k); if (k * k + 1 < (1ull << 32)) ok32(k * k + 1); }
  for (u64 v = 0xFFFFFFFFull - 4096; v <= 0xFFFFFFFFull; ++v) ok32(v);
  // 64-bit: values from the command line, one per line of stdin
  unsigned long long x;
  while (scanf("%llu", &x) == 1) printf("%lld\n", (long long)lego_isqrt((i64)x));
  fprintf(stderr, "bad32 %llu\n", bad);
  return bad != 0;
}
"""


def test_integer_square_root_of_generated_code():
    """The exact integer square root the kernels use (the antidiagonal GenP,
    Figure 7 with an exact root): 32-bit operands at every perfect-square
    boundary, 64-bit ones against math.isqrt on sampled values."""
    import math
    import random
    import paper_2505_08091_amd as L
    src = L.plan_source("apply", L.as_layout(L.GenP("antidiag", [64, 64])), param=4)
    rng = random.Random(5)
    vals = [0, 1, 2, 3, (1 << 62) - 1, 1 << 62, (1 << 63) - 1] + [rng.randrange(1 << 63) for _ in range(2000)]
    vals += [k * k + d for k in (rng.randrange(1 << 31) for _ in range(500)) for d in (-1, 0, 1)]
    with tempfile.TemporaryDirectory() as tmp:
        head = src.split(MARK)[0]
        cpp, exe = os.path.join(tmp, "s.cpp"), os.path.join(tmp, "s")
        with open(cpp, "w") as f:
            f.write(HARNESS_COMMON + head + HARNESS_ISQRT)
        r = subprocess.run(["g++", "-O2", "-std=c++17", "-w", cpp, "-o", exe], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-4000:]
        r = subprocess.run([exe], input="\n".join(map(str, vals)), capture_output=True, text=True, timeout=120)
        assert r.returncode == 0, r.stderr
        got = [int(t) for t in r.stdout.split()]
        assert got == [math.isqrt(v) for v in vals]
