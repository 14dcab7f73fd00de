// Layout remap kernels: dst[p] = src[M(p)] with M = L_src.apply o L_dst.inv.
// Generated code defines, before this text:
//   ELEM_T     unsigned integer type of the element size (bytes are copied)
//   IDX_T      index type of the generated functions
// Direct path (M keeps runs of at least V elements):
//   V, NVEC, NT, UNROLL
//   LEGO_FN IDX_T src_vec(IDX_T t)   source vector index of destination vector t
//   LEGO_FN IDX_T blk(IDX_T b)       destination chunk of schedule position b
//   NBLK                             number of chunks
//   SRC_SEP, LEGO_FN IDX_T src_base(IDX_T c), src_loc(IDX_T r)   1: the source
//                                    vector of chunk c's vector r is src_base(c) + src_loc(r)
//   MASKED, LEGO_FN IDX_T src_ok(IDX_T t)   1: vector t has a source (an
//                                    ExpandBy source, Figure 9); else it is zero
// LDS path (both sides are digit permutations; a tile of TILE elements is read
// in source order into LDS and written in destination order):
//   TILE, NT, VL, VS, LDSW_CONTIG, LDS_BLOCK
//   LEGO_FN IDX_T src_off(IDX_T g, IDX_T q)   element offset of source-side vector q of tile g
//   LEGO_FN IDX_T ldsw(IDX_T q, IDX_T e)      LDS slot of element e of that vector
//   LDS_BLOCK 1 (a transposing tile): a thread moves blocks of NX source
//   vectors that hold NY whole destination vectors; then instead
//   LEGO_FN IDX_T src_off(IDX_T g, IDX_T b, IDX_T x)  offset of load x of block b
//   LEGO_FN IDX_T ldsw(IDX_T b, IDX_T y)      LDS slot of destination vector y of block b
//   LEGO_FN int blk_el(int k)                 element k of destination vector k / VS
//                                             is element blk_el(k) of the block's loads
//   LEGO_FN IDX_T ldsr(IDX_T q)               LDS slot of destination-side vector q
//   LEGO_FN IDX_T dst_off(IDX_T g, IDX_T q)   element offset of destination-side vector q
// Box path (2-D maps without digit structure): a BX x BX box of the logical
// index space is read line by line in one kind of line and written in another,
// through LDS:
//   BX, BPAD, NBR x NBC (the grid of boxes), EXT0, EXT1 (logical extents), NT
//   S_ORD, D_ORD     kind of line of the load and store sides (0 rows, 1
//                    columns, 2 pairs of antidiagonals of the box)
//   LEGO_FN void bord(IDX_T b, IDX_T* bi, IDX_T* bj)  box of workgroup b
//   S_SEP, LEGO_FN IDX_T s_u(IDX_T bi, IDX_T bj, IDX_T r), s_l(IDX_T l)   1: the
//                    source offset of lane l on row, column or antidiagonal r
//                    of box (bi, bj) is s_u(bi, bj, r) + s_l(l); 0: LEGO_FN
//                    IDX_T s_f(IDX_T i, IDX_T j) of logical point (i, j)
//   D_SEP, d_u, d_l, d_f  the same for the destination
// NONTEMPORAL: bit 0 streams (non-temporal) global loads, bit 1 stores.

#if NONTEMPORAL & 1
#define LEGO_LD(p) __builtin_nontemporal_load(p)
#else
#define LEGO_LD(p) (*(p))
#endif
#if NONTEMPORAL & 2
#define LEGO_ST(v, p) __builtin_nontemporal_store((v), (p))
#else
#define LEGO_ST(v, p) (*(p) = (v))
#endif

#ifdef LEGO_REMAP_DIRECT
typedef ELEM_T vec_t __attribute__((ext_vector_type(V)));
// Copies destination chunk c (NT*UNROLL vectors): UNROLL loads in flight per
// thread, then UNROLL stores.
LEGO_FN void remap_chunk(const vec_t* __restrict__ src, vec_t* __restrict__ dst, u64 c) {
  const u64 base = c * (NT * UNROLL) + threadIdx.x;
#if SRC_SEP
  // chunk part of the map, once per workgroup (c is uniform)
  const vec_t* __restrict__ sc = src + src_base((IDX_T)c);
#define SRC_OF(t, u) (sc + src_loc((IDX_T)((u64)(u) * NT + threadIdx.x)))
#else
#define SRC_OF(t, u) (src + src_vec((IDX_T)(t)))
#endif
  vec_t v[UNROLL];
  if ((c + 1) * (NT * UNROLL) <= NVEC) {
    // A whole chunk (every chunk but a ragged last one): no bounds tests, so
    // the UNROLL loads are issued back to back.  A vector without a source
    // reads the buffer's first vector instead and is zeroed, keeping the
    // loads free of branches.
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const u64 t = base + (u64)u * NT;
#if MASKED
      const bool ok = src_ok((IDX_T)t);
      const vec_t x = LEGO_LD(ok ? SRC_OF(t, u) : src);
      v[u] = ok ? x : (vec_t){};
#else
      v[u] = LEGO_LD(SRC_OF(t, u));
#endif
    }
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) LEGO_ST(v[u], dst + base + (u64)u * NT);
    return;
  }
#pragma unroll
  for (int u = 0; u < UNROLL; ++u) {
    const u64 t = base + (u64)u * NT;
#if MASKED
    if (t < NVEC) v[u] = src_ok((IDX_T)t) ? LEGO_LD(SRC_OF(t, u)) : (vec_t){};
#else
    if (t < NVEC) v[u] = LEGO_LD(SRC_OF(t, u));
#endif
  }
#undef SRC_OF
#pragma unroll
  for (int u = 0; u < UNROLL; ++u) {
    const u64 t = base + (u64)u * NT;
    if (t < NVEC) LEGO_ST(v[u], dst + t);
  }
}
// Workgroup b handles destination chunks blk(b), blk(b + G), ... (G = the
// grid size; NBLK chunks in all).  The chunk order is a layout chosen so that
// the workgroups resident at one time touch spread-out source addresses.
extern "C" __global__ __launch_bounds__(NT) void lego_remap_direct(const vec_t* __restrict__ src,
                                                                   vec_t* __restrict__ dst) {
  for (u64 b = blockIdx.x; b < NBLK; b += gridDim.x) remap_chunk(src, dst, (u64)blk((IDX_T)b));
}
#endif

#ifdef LEGO_REMAP_LDS
typedef ELEM_T vl_t __attribute__((ext_vector_type(VL)));
typedef ELEM_T vs_t __attribute__((ext_vector_type(VS)));
extern "C" __global__ __launch_bounds__(NT) void lego_remap_lds(const ELEM_T* __restrict__ src,
                                                                ELEM_T* __restrict__ dst) {
  __shared__ ELEM_T tile[TILE];
  const IDX_T g = blockIdx.x;
#if LDS_BLOCK
  // Source-order phase by blocks: NX coalesced vector reads per block, a
  // permutation in registers, NY whole destination vectors written to LDS.
  vl_t v[TILE / (VL * NX) / NT][NX];
#pragma unroll
  for (int it = 0; it < TILE / (VL * NX) / NT; ++it) {
    const IDX_T b = it * NT + threadIdx.x;
#pragma unroll
    for (int x = 0; x < NX; ++x) v[it][x] = LEGO_LD((const vl_t*)(src + src_off(g, b, (IDX_T)x)));
  }
#pragma unroll
  for (int it = 0; it < TILE / (VL * NX) / NT; ++it) {
    const IDX_T b = it * NT + threadIdx.x;
#pragma unroll
    for (int y = 0; y < NY; ++y) {
      vs_t w;
#pragma unroll
      for (int e = 0; e < VS; ++e) w[e] = v[it][blk_el(y * VS + e) / VL][blk_el(y * VS + e) % VL];
      *(vs_t*)&tile[ldsw(b, (IDX_T)y)] = w;
    }
  }
#else
  // Source-order phase: coalesced vector reads, scattered LDS writes.
  vl_t v[TILE / VL / NT];
#pragma unroll
  for (int it = 0; it < TILE / VL / NT; ++it) {
    const IDX_T q = it * NT + threadIdx.x;
    v[it] = LEGO_LD((const vl_t*)(src + src_off(g, q)));
  }
#pragma unroll
  for (int it = 0; it < TILE / VL / NT; ++it) {
    const IDX_T q = it * NT + threadIdx.x;
#if LDSW_CONTIG
    *(vl_t*)&tile[ldsw(q, 0)] = v[it];
#else
#pragma unroll
    for (int e = 0; e < VL; ++e) tile[ldsw(q, e)] = v[it][e];
#endif
  }
#endif
  __syncthreads();
  // Destination-order phase: vector LDS reads, coalesced vector writes.
#pragma unroll
  for (int it = 0; it < TILE / VS / NT; ++it) {
    const IDX_T q = it * NT + threadIdx.x;
    const vs_t w = *(const vs_t*)&tile[ldsr(q)];
    LEGO_ST(w, (vs_t*)(dst + dst_off(g, q)));
  }
}
#endif

#ifdef LEGO_REMAP_BOX
// One workgroup (NT threads, NT/64 waves) per BX x BX box of the logical
// index space (BX = 64 or 128), staged through LDS.  Each side is copied line
// by line; lane l of a wave takes positions x = l, l + 64, ... (EPL of them)
// of line p of the box, a line being
//   ORD 0: box row p:    (a, b) = (p, x),
//   ORD 1: box column p: (a, b) = (x, p),
//   ORD 2: box antidiagonals p and p + BX together (their lengths add up to
//          BX): (a, b) = (x, (p - x) mod BX), on antidiagonal p for x <= p
//          and on antidiagonal p + BX for x > p, so every position is used.
// Wave w copies lines w, w + NT/64, ...  Where the planner split a side's
// element offset into a part of (box, row or column or antidiagonal r) and a
// part of the position x (S_SEP, D_SEP), an element costs one add: the parts
// of every r are computed once per box, r = 64k + q in lane q of table k, and
// read out of that lane for each line; otherwise the offset is s_f(i, j) of
// the point.  Points past the logical extents (boxes on the last row or
// column) are neither read nor written.  Each LDS row is BX + BPAD elements,
// the pad chosen against bank conflicts of both kinds of line.
#define NW (NT / 64)
#define EPL (BX / 64)
#define NITER (BX / NW)
#define NTAB(o) ((o) == 2 ? 2 * EPL : EPL)
template <bool B>
struct lego_flag {
  static constexpr bool value = B;
};
// Lane q's value of x (x holds one value per lane).
LEGO_FN IDX_T lane_read(IDX_T x, IDX_T q) {
  if (sizeof(IDX_T) == 8) {
    const u64 v = (u64)x;
    const u32 lo = (u32)__builtin_amdgcn_readlane((int)(u32)v, (int)q);
    const u32 hi = (u32)__builtin_amdgcn_readlane((int)(u32)(v >> 32), (int)q);
    return (IDX_T)(((u64)hi << 32) | lo);
  }
  return (IDX_T)(u32)__builtin_amdgcn_readlane((int)x, (int)q);
}
template <int ORD>
LEGO_FN void box_pt(IDX_T p, IDX_T x, IDX_T* a, IDX_T* b) {
  if (ORD == 0) {
    *a = p;
    *b = x;
  } else if (ORD == 1) {
    *a = x;
    *b = p;
  } else {
    *a = x;
    *b = (p - x) & (BX - 1);
  }
}
// Offset of position x = l + 64 e of line p (it-th line of this wave) of a
// side whose offset is split: the part of its row, column or antidiagonal,
// read out of its lane of the tables, plus the position's part.
template <int ORD>
LEGO_FN IDX_T line_off(const IDX_T* tab, const IDX_T* xpart, int it, int e, IDX_T p, IDX_T x) {
  const int k = it * NW / 64;  // p / 64: every line of one iteration is in one table
  const IDX_T q = p % 64u;
  if (ORD == 2) {
    const IDX_T lo = lane_read(tab[k], q), hi = lane_read(tab[k + EPL], q);
    return (x <= p ? lo : hi) + xpart[e];
  }
  return lane_read(tab[k], q) + xpart[e];
}
extern "C" __global__ __launch_bounds__(NT) void lego_remap_box(const ELEM_T* __restrict__ src,
                                                                ELEM_T* __restrict__ dst) {
  __shared__ ELEM_T tile[BX * (BX + BPAD)];
  IDX_T bi, bj;
  bord((IDX_T)blockIdx.x, &bi, &bj);
  const IDX_T i0 = bi * BX, j0 = bj * BX;
  const bool whole = i0 + BX <= EXT0 && j0 + BX <= EXT1;
  const IDX_T l = threadIdx.x % 64u;
  const IDX_T w = __builtin_amdgcn_readfirstlane(threadIdx.x / 64u);
#if S_SEP
  IDX_T s_tab[NTAB(S_ORD)], s_x[EPL];
#pragma unroll
  for (int k = 0; k < NTAB(S_ORD); ++k) s_tab[k] = s_u(bi, bj, 64u * k + l);
#pragma unroll
  for (int e = 0; e < EPL; ++e) s_x[e] = s_l(l + 64u * e);
#endif
#if D_SEP
  IDX_T d_tab[NTAB(D_ORD)], d_x[EPL];
#pragma unroll
  for (int k = 0; k < NTAB(D_ORD); ++k) d_tab[k] = d_u(bi, bj, 64u * k + l);
#pragma unroll
  for (int e = 0; e < EPL; ++e) d_x[e] = d_l(l + 64u * e);
#endif
  // All loads first, NITER * EPL in flight per thread; boxes inside the
  // extents (all but the last row and column of boxes) without any test.
  ELEM_T v[NITER][EPL];
  auto load = [&](auto checked) {
#pragma unroll
    for (int it = 0; it < NITER; ++it)
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const IDX_T p = (IDX_T)it * NW + w, x = l + 64u * e;
        IDX_T a, b;
        box_pt<S_ORD>(p, x, &a, &b);
        if (decltype(checked)::value && !(i0 + a < EXT0 && j0 + b < EXT1)) continue;
#if S_SEP
        v[it][e] = LEGO_LD(src + line_off<S_ORD>(s_tab, s_x, it, e, p, x));
#else
        v[it][e] = LEGO_LD(src + s_f(i0 + a, j0 + b));
#endif
      }
  };
  if (whole) load(lego_flag<false>{});
  else load(lego_flag<true>{});
#pragma unroll
  for (int it = 0; it < NITER; ++it)
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      const IDX_T p = (IDX_T)it * NW + w, x = l + 64u * e;
      IDX_T a, b;
      box_pt<S_ORD>(p, x, &a, &b);
      tile[a * (BX + BPAD) + b] = v[it][e];
    }
  __syncthreads();
  auto store = [&](auto checked) {
#pragma unroll
    for (int it = 0; it < NITER; ++it)
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const IDX_T p = (IDX_T)it * NW + w, x = l + 64u * e;
        IDX_T a, b;
        box_pt<D_ORD>(p, x, &a, &b);
        if (decltype(checked)::value && !(i0 + a < EXT0 && j0 + b < EXT1)) continue;
#if D_SEP
        LEGO_ST(tile[a * (BX + BPAD) + b], dst + line_off<D_ORD>(d_tab, d_x, it, e, p, x));
#else
        LEGO_ST(tile[a * (BX + BPAD) + b], dst + d_f(i0 + a, j0 + b));
#endif
      }
  };
  if (whole) store(lego_flag<false>{});
  else store(lego_flag<true>{});
}
#undef NTAB
#undef NITER
#undef EPL
#undef NW
#endif
