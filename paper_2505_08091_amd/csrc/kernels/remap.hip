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
//   TILE, NT, VL, VS, LDSW_CONTIG
//   LEGO_FN IDX_T src_off(IDX_T g, IDX_T q)   element offset of source-side vector q of tile g
//   LEGO_FN IDX_T ldsw(IDX_T q, IDX_T e)      LDS slot of element e of that vector
//   LEGO_FN IDX_T ldsr(IDX_T q)               LDS slot of destination-side vector q
//   LEGO_FN IDX_T dst_off(IDX_T g, IDX_T q)   element offset of destination-side vector q
// Box path (2-D maps without digit structure): a BR x BC box of the logical
// index space is read in one order and written in another, through LDS:
//   BR, BC, BPAD, NBR x NBC (the grid of boxes), EXT0, EXT1 (logical extents), NT
//   LEGO_FN void bord(IDX_T b, IDX_T* bi, IDX_T* bj)  box of workgroup b
//   LEGO_FN void ws(IDX_T q, IDX_T* a, IDX_T* b)   box element read q-th
//   LEGO_FN void wd(IDX_T q, IDX_T* a, IDX_T* b)   box element written q-th
//   LEGO_FN IDX_T bsrc(IDX_T i, IDX_T j), bdst(IDX_T i, IDX_T j)   element
//                                    offsets of logical point (i, j)
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
// One workgroup per box.  The read order makes consecutive lanes read
// consecutive source addresses, the write order consecutive destination
// addresses (runs of up to a box side); each LDS row is BC + BPAD elements,
// the pad chosen so that neither order puts two lanes of a wave on one bank.
// Points past the logical extents (boxes on the last row or column) are
// neither read nor written.
#define BOX (BR * BC)
extern "C" __global__ __launch_bounds__(NT) void lego_remap_box(const ELEM_T* __restrict__ src,
                                                                ELEM_T* __restrict__ dst) {
  __shared__ ELEM_T tile[BR * (BC + BPAD)];
  IDX_T bi, bj;
  bord((IDX_T)blockIdx.x, &bi, &bj);
  const IDX_T i0 = bi * BR, j0 = bj * BC;
  const bool whole = i0 + BR <= EXT0 && j0 + BC <= EXT1;
  ELEM_T v[BOX / NT];
  IDX_T slot[BOX / NT];
  // All reads first, so that BOX / NT loads per thread are in flight at once.
#pragma unroll
  for (int u = 0; u < BOX / NT; ++u) {
    IDX_T a, b;
    ws((IDX_T)(u * NT + threadIdx.x), &a, &b);
    slot[u] = a * (BC + BPAD) + b;
    if (whole || (i0 + a < EXT0 && j0 + b < EXT1)) v[u] = LEGO_LD(src + bsrc(i0 + a, j0 + b));
  }
#pragma unroll
  for (int u = 0; u < BOX / NT; ++u) tile[slot[u]] = v[u];
  __syncthreads();
#pragma unroll
  for (int u = 0; u < BOX / NT; ++u) {
    IDX_T a, b;
    wd((IDX_T)(u * NT + threadIdx.x), &a, &b);
    if (whole || (i0 + a < EXT0 && j0 + b < EXT1)) LEGO_ST(tile[a * (BC + BPAD) + b], dst + bdst(i0 + a, j0 + b));
  }
}
#undef BOX
#endif
