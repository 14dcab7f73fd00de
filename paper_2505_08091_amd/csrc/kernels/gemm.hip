// Hierarchically tiled GEMM on the gfx950 matrix cores: C = A * B, fp16/bf16
// inputs, fp32 accumulation, fp32 C.  Every index comes from a layout:
//   - the workgroup -> (tm, tn) tile schedule (grouped order, XCD remap),
//   - the operand layouts of A, B and C in global memory,
//   - the thread -> element map of the global-to-LDS copy,
//   - the LDS tile layouts (XOR swizzles that keep 16-byte vectors whole),
//   - the MFMA fragment layouts (lane, element) -> (row, k) and (row, col).
// The generated code defines, before this text:
//   BM BN BK         workgroup tile
//   MB KB            MFMA block (32x32x16 or 16x16x32)
//   MI NI            MFMA blocks per wave along m and n
//   MI_LIVE NI_LIVE  the leading blocks of these that hold some element of C
//                    (fewer only where M or N is below one tile)
//   NWAVES NT KT     waves per workgroup, threads (64 * NWAVES), K / BK
//   IN_BF16          1: bf16 inputs, 0: fp16
//   A_NV A_V A_SEP A_SVEC A_FRVEC A_NVEC A_GUARD (and B_*): vectors per thread
//       per K step, elements per vector, additively separable global offset,
//       vector LDS store, vector fragment read, vectors per tile, and whether
//       the last round of vectors covers only part of the threads
//   C_SEP
//   STORE_AT         k-substep during which the next tile is written to LDS
//   PREFETCH         1 or 2: K steps between a tile's global load and its use
//   ROLLING          1: register-staged loads use the rolling pipeline
//   DIRECT_LDS       1: global-to-LDS copies without registers, NSTAGES-deep ring
//   NSTAGES          LDS stages (2 unless DIRECT_LDS)
//   sched(pid, &tm, &tn)
//   a_gt(tm) a_gk(kt) a_gl(tid, u)   or   a_gf(tm, kt, tid, u)
//   a_s(tid, u, e)                   LDS element offset of element e of load vector u
//   a_fr(lane, w, mi, s, e)          LDS element offset of fragment element e
//   A_FRTR, a_ft(lane, w, mi, s, h)  fragments read with the transposing LDS
//                                    load: the address lane supplies for half h
//   A_FRDW                           fragments read as 4 dwords at a_fr(.., 2p),
//                                    elements 2p and 2p + 1 adjacent in LDS;
//   A_FRDW_D, a_fd(lane, w, mi, s, h)  with A_FRDW_D > 0, dword 2h at a_fd(h)
//                                    and dword 2h + 1 A_FRDW_D elements on
//   A_FRZP, a_fz(lane, w, m, s, h)   MFMA blocks 2m, 2m+1 hold the even and odd
//                                    rows of a band; a lane reads both from two
//                                    16-byte slots at a_fz(h), h = 0, 1
//   (b_* likewise with tn)
//   c_t(tm, tn) c_l(lane, w, mi, ni, r)   or   c_f(tm, tn, lane, w, mi, ni, r)
//   A_BUF (and B_BUF): direct copies are range-checked buffer loads with
//       32-bit byte offsets (operands under 2 GiB; 0.5% faster than global
//       loads on the 8192^3 bf16 GEMM, and fewer address registers)
//   A_EDGE, a_ok(tm, kt, tid, u), A_BYTES (and B_*): tiles padded past the
//       operand (Section III-D partial tiles): load vector u is inside (1) or
//       padding (0, read as zero); the operand's size in bytes
//   C_EDGE, c_ok(tm, tn, lane, w, mi, ni, r): the C element exists
//   A_VR A_VC A_BIDX (and B_*): a load vector that is an A_VR x A_VC block of
//       the tile; A_BIDX[r * A_VC + c] is the vector element at block (r, c),
//       and each block row is stored to LDS as one A_VC-element vector

typedef unsigned short elem_t;
typedef elem_t av_t __attribute__((ext_vector_type(A_V)));
typedef elem_t bv_t __attribute__((ext_vector_type(B_V)));
typedef elem_t e8_t __attribute__((ext_vector_type(8)));
#if IN_BF16
typedef __bf16 mf_t __attribute__((ext_vector_type(8)));
#else
typedef _Float16 mf_t __attribute__((ext_vector_type(8)));
#endif
#if MB == 32
typedef float acc_t __attribute__((ext_vector_type(16)));
#define NREG 16
#if IN_BF16
#define MFMA(a, b, c) __builtin_amdgcn_mfma_f32_32x32x16_bf16((a), (b), (c), 0, 0, 0)
#else
#define MFMA(a, b, c) __builtin_amdgcn_mfma_f32_32x32x16_f16((a), (b), (c), 0, 0, 0)
#endif
#else
typedef float acc_t __attribute__((ext_vector_type(4)));
#define NREG 4
#if IN_BF16
#define MFMA(a, b, c) __builtin_amdgcn_mfma_f32_16x16x32_bf16((a), (b), (c), 0, 0, 0)
#else
#define MFMA(a, b, c) __builtin_amdgcn_mfma_f32_16x16x32_f16((a), (b), (c), 0, 0, 0)
#endif
#endif

#define A_STAGE (BM * BK)
#define B_STAGE (BN * BK)
#define STAGE (A_STAGE + B_STAGE)

LEGO_FN mf_t lds_frag(const elem_t* base, IDX_T off) {
  return __builtin_bit_cast(mf_t, *(const e8_t*)(base + off));
}
// Fragment as 4 dwords, each 2 consecutive k of the lane's row (Z-order
// operands, whose LDS slots interleave two rows); reads whose offsets differ
// by a constant pair up into ds_read2_b32.
typedef unsigned u4_t __attribute__((ext_vector_type(4)));
LEGO_FN mf_t lds_frag_dw(const elem_t* base, IDX_T o0, IDX_T o1, IDX_T o2, IDX_T o3) {
  const u4_t t = {*(const unsigned*)(base + o0), *(const unsigned*)(base + o1), *(const unsigned*)(base + o2),
                  *(const unsigned*)(base + o3)};
  return __builtin_bit_cast(mf_t, t);
}

// Fragment through two transposing LDS loads (ds_read_b64_tr_b16): elements
// 0-3 from the addresses of half 0, elements 4-7 from those of half 1.  With
// direct global-to-LDS copies the loads are issued as inline assembly: the
// compiler's own form of this load is ordered behind every direct copy in
// flight (a full vmcnt wait before each read), which would serialize the
// copies with the MFMAs.  The compiler does not track these loads, so
// FRAG_WAIT below waits for them before their fragments are used and before
// every barrier.  Register-staged plans have no such copies and use the
// compiler's form.
typedef short s4_t __attribute__((ext_vector_type(4)));
LEGO_FN s4_t lds_read_tr(const elem_t* p) {
#if DIRECT_LDS
  s4_t r;
  const unsigned a = (unsigned)(unsigned long)(__attribute__((address_space(3))) const void*)p;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(r) : "v"(a));
  return r;
#else
  // No global-to-LDS copies in flight: the compiler's own (tracked) form.
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4_t*)p);
#endif
}
LEGO_FN mf_t lds_frag_tr(const elem_t* base, IDX_T off0, IDX_T off1) {
  const s4_t lo = lds_read_tr(base + off0);
  const s4_t hi = lds_read_tr(base + off1);
  const e8_t t = {(elem_t)lo[0], (elem_t)lo[1], (elem_t)lo[2], (elem_t)lo[3],
                  (elem_t)hi[0], (elem_t)hi[1], (elem_t)hi[2], (elem_t)hi[3]};
  return __builtin_bit_cast(mf_t, t);
}
#if A_FRTR || B_FRTR
// s_waitcnt lgkmcnt(0) (vmcnt and expcnt at their maxima), then no motion
// across it.
#define FRAG_WAIT()                         \
  do {                                      \
    __builtin_amdgcn_s_waitcnt(0xC07F);     \
    __builtin_amdgcn_sched_barrier(0);      \
  } while (0)
// Start of a substep of the direct-copy loop: the fragments of this substep
// must have arrived, those of the FRAG_DIST - 1 substeps after it may still
// be in flight.  A wave's LDS operations complete in issue order, and at
// least FRAG_READS of them were issued per substep after this substep's last
// read, so waiting until at most (FRAG_DIST - 1) * FRAG_READS (the counter
// holds 15) are outstanding is enough.
#define LGKM_NEXT ((FRAG_DIST - 1) * FRAG_READS < 15 ? (FRAG_DIST - 1) * FRAG_READS : 15)
#define FRAG_WAIT_NEXT()                                  \
  do {                                                    \
    __builtin_amdgcn_s_waitcnt(0xC07F | (LGKM_NEXT << 8)); \
    __builtin_amdgcn_sched_barrier(0);                    \
  } while (0)
#else
#define FRAG_WAIT() \
  do {              \
  } while (0)
#define FRAG_WAIT_NEXT() FRAG_WAIT()
#endif
// Fragment register sets: FRAG_DIST + 1, or one per substep when that does
// not divide the substeps of a step (a set's index must repeat every step).
#ifndef FRAG_DIST
#define FRAG_DIST 1
#endif
// MFMA rows after the stage barrier over which the copies of a step are
// spread.
#ifndef FRAG_SPREAD
#define FRAG_SPREAD 0
#endif
#ifndef DMA_ROWS
#define DMA_ROWS (FRAG_DIST * MFMA_ROWS)
#endif
#if (BK / KB) % (FRAG_DIST + 1) == 0
#define NFB (FRAG_DIST + 1)
#else
#define NFB (BK / KB)
#endif
// The reads of substep s + FRAG_DIST must go to another set than substep s
// uses: FRAG_DIST + 1 sets at least, which needs more substeps than
// FRAG_DIST.
static_assert(FRAG_DIST == 1 || (FRAG_DIST < BK / KB && NFB > FRAG_DIST), "fragment sets");
// LDS read instructions per fragment.
#define A_FRD (A_FRTR ? 2 : (A_FRVEC || A_FRZP ? 1 : (A_FRDW ? 2 : 8)))
#define B_FRD (B_FRTR ? 2 : (B_FRVEC ? 1 : (B_FRDW ? 2 : 8)))
#define FRAG_READS (MI_LIVE * A_FRD + NI_LIVE * B_FRD)

template <bool B>
struct lego_bool {
  static constexpr bool value = B;
};

extern "C" __global__ __launch_bounds__(NT) void lego_gemm(const elem_t* __restrict__ A, const elem_t* __restrict__ B,
                                                           float* __restrict__ C) {
  __shared__ __attribute__((aligned(16))) elem_t lds[NSTAGES * STAGE];
  const IDX_T tid = threadIdx.x;
  const IDX_T lane = tid % 64u;
  const IDX_T w = tid / 64u;
  IDX_T tm, tn;
  sched((IDX_T)blockIdx.x, &tm, &tn);

#if A_SEP
  const elem_t* __restrict__ Ab = A + a_gt(tm);
  IDX_T a_loc[A_NV];
#pragma unroll
  for (int u = 0; u < A_NV; ++u) a_loc[u] = a_gl(tid, u);
#endif
#if B_SEP
  const elem_t* __restrict__ Bb = B + b_gt(tn);
  IDX_T b_loc[B_NV];
#pragma unroll
  for (int u = 0; u < B_NV; ++u) b_loc[u] = b_gl(tid, u);
#endif

  // Global-to-LDS staging registers.  With PREFETCH == 2 there are two sets:
  // the tile for step kt+2 is loaded while the tile for step kt+1 (loaded one
  // step earlier) is written to LDS, hiding more than a full step of memory
  // latency.
#if (PREFETCH == 2 || ROLLING) && BK / KB >= 2
#define NSETS 1  // the rolling pipeline below reuses one set
#else
#define NSETS PREFETCH
#endif
  av_t ra[NSETS][A_NV];
  bv_t rb[NSETS][B_NV];
  acc_t acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j) acc[i][j] = (acc_t){};
  // The accumulators of tile (tm_, tn_) to C, with non-temporal stores (C is
  // not read again; measured ahead of ordinary stores).  Each store writes
  // 2 rows of 32 consecutive C elements of an MFMA block (the 32x32 C
  // fragment layout); 16-byte stores of 4 consecutive elements from
  // operand-swapped MFMAs write 32-byte pieces of 32 rows and measured 20%
  // slower on the 8192^3 bf16 GEMM.
  auto store_c = [&](IDX_T tm_, IDX_T tn_) {
    // The tile's offset is opaque to the compiler: with one tile it is a
    // constant, and the compiler then built all 256 store addresses of a
    // lane ahead of the k-loop (512 VGPRs) and spilled them.  (An integer, so
    // that C keeps its global address space and the stores stay global
    // stores, which do not count against the LDS wait counter.)
#if C_SEP
    IDX_T ct = c_t(tm_, tn_);
    asm volatile("" : "+v"(ct));
    float* __restrict__ Cb = C + ct;
#else
    IDX_T ct = 0;
    asm volatile("" : "+v"(ct));
    float* __restrict__ Cb = C + ct;
#endif
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NI; ++j)
#pragma unroll
        for (int r = 0; r < NREG; ++r) {
#if C_EDGE
          if (!c_ok(tm_, tn_, lane, w, i, j, r)) continue;
#endif
#if C_SEP
          __builtin_nontemporal_store(acc[i][j][r], Cb + c_l(lane, w, i, j, r));
#else
          __builtin_nontemporal_store(acc[i][j][r], Cb + c_f(tm_, tn_, lane, w, i, j, r));
#endif
        }
  };

  // Load vectors [lo, hi) of the tile for step kt (A's A_NV vectors, then
  // B's B_NV) into staging set rbuf.
  auto gload_part = [&](IDX_T kt, int rbuf, int lo, int hi) {
#pragma unroll
    for (int u = 0; u < A_NV; ++u) {
      if (u < lo || u >= hi) continue;
      if (A_GUARD && (IDX_T)u * NT + tid >= A_NVEC) continue;
#if A_EDGE
      if (!a_ok(tm, kt, tid, u)) {
        ra[rbuf][u] = (av_t){};
        continue;
      }
#endif
#if A_SEP
      ra[rbuf][u] = *(const av_t*)(Ab + a_gk(kt) + a_loc[u]);
#else
      ra[rbuf][u] = *(const av_t*)(A + a_gf(tm, kt, tid, u));
#endif
    }
#pragma unroll
    for (int u = 0; u < B_NV; ++u) {
      if (A_NV + u < lo || A_NV + u >= hi) continue;
      if (B_GUARD && (IDX_T)u * NT + tid >= B_NVEC) continue;
#if B_EDGE
      if (!b_ok(tn, kt, tid, u)) {
        rb[rbuf][u] = (bv_t){};
        continue;
      }
#endif
#if B_SEP
      rb[rbuf][u] = *(const bv_t*)(Bb + b_gk(kt) + b_loc[u]);
#else
      rb[rbuf][u] = *(const bv_t*)(B + b_gf(tn, kt, tid, u));
#endif
    }
  };
  auto gload = [&](IDX_T kt, int rbuf) { gload_part(kt, rbuf, 0, A_NV + B_NV); };
  // Write vectors [lo, hi) of staging set rbuf to LDS stage `stage`.
  auto sstore_part = [&](int stage, int rbuf, int lo, int hi) {
    elem_t* la = lds + stage * STAGE;
    elem_t* lb = la + A_STAGE;
#pragma unroll
    for (int u = 0; u < A_NV; ++u) {
      if (u < lo || u >= hi) continue;
      if (A_GUARD && (IDX_T)u * NT + tid >= A_NVEC) continue;
#if A_VR > 1 && A_SVEC
      typedef elem_t ar_t __attribute__((ext_vector_type(A_VC)));
#pragma unroll
      for (int r = 0; r < A_VR; ++r) {
        ar_t piece;
#pragma unroll
        for (int c = 0; c < A_VC; ++c) piece[c] = ra[rbuf][u][A_BIDX[r * A_VC + c]];
        *(ar_t*)(la + a_s(tid, u, A_BIDX[r * A_VC])) = piece;
      }
#elif A_SVEC
      *(av_t*)(la + a_s(tid, u, 0)) = ra[rbuf][u];
#else
#pragma unroll
      for (int e = 0; e < A_V; ++e) la[a_s(tid, u, e)] = ra[rbuf][u][e];
#endif
    }
#pragma unroll
    for (int u = 0; u < B_NV; ++u) {
      if (A_NV + u < lo || A_NV + u >= hi) continue;
      if (B_GUARD && (IDX_T)u * NT + tid >= B_NVEC) continue;
#if B_VR > 1 && B_SVEC
      typedef elem_t br_t __attribute__((ext_vector_type(B_VC)));
#pragma unroll
      for (int r = 0; r < B_VR; ++r) {
        br_t piece;
#pragma unroll
        for (int c = 0; c < B_VC; ++c) piece[c] = rb[rbuf][u][B_BIDX[r * B_VC + c]];
        *(br_t*)(lb + b_s(tid, u, B_BIDX[r * B_VC])) = piece;
      }
#elif B_SVEC
      *(bv_t*)(lb + b_s(tid, u, 0)) = rb[rbuf][u];
#else
#pragma unroll
      for (int e = 0; e < B_V; ++e) lb[b_s(tid, u, e)] = rb[rbuf][u][e];
#endif
    }
  };

  auto sstore = [&](int stage, int rbuf) { sstore_part(stage, rbuf, 0, A_NV + B_NV); };

  // Fragments of one k-substep, double-buffered in registers: the reads of
  // substep s+1 are in flight while the MFMAs of substep s run.
  mf_t af[NFB][MI], bf[NFB][NI];
  // Fragments [lo, hi) of substep s into set buf: A's MI fragments, then
  // B's NI.
  auto fload_part = [&](const elem_t* la, const elem_t* lb, int s, int buf, int lo, int hi) {
#pragma unroll
    for (int i = 0; i < MI; ++i) {
      if (i < lo || i >= hi || i >= MI_LIVE) continue;
#if A_FRTR
      af[buf][i] = lds_frag_tr(la, a_ft(lane, w, i, s, 0), a_ft(lane, w, i, s, 1));
#elif A_FRVEC
      af[buf][i] = lds_frag(la, a_fr(lane, w, i, s, 0));
#elif A_FRZP
      // Row pairs: blocks i and i + 1 hold the even and the odd rows of a
      // band, and two 16-byte reads bring a lane both rows' 8 k (a slot is
      // one 2 x 4 Z block); the registers keep the slots as read (a_op picks
      // the operands).  The odd block is read with its even partner.
      if (i % 2 == 0) {
        af[buf][i] = lds_frag(la, a_fz(lane, w, i / 2, s, 0));
        af[buf][i + 1] = lds_frag(la, a_fz(lane, w, i / 2, s, 1));
      }
#elif A_FRDW && A_FRDW_D
      {
        const IDX_T o0 = a_fd(lane, w, i, s, 0), o1 = a_fd(lane, w, i, s, 1);
        af[buf][i] = lds_frag_dw(la, o0, o0 + A_FRDW_D, o1, o1 + A_FRDW_D);
      }
#elif A_FRDW
      af[buf][i] = lds_frag_dw(la, a_fr(lane, w, i, s, 0), a_fr(lane, w, i, s, 2), a_fr(lane, w, i, s, 4),
                               a_fr(lane, w, i, s, 6));
#else
      e8_t t;
#pragma unroll
      for (int e = 0; e < 8; ++e) t[e] = la[a_fr(lane, w, i, s, e)];
      af[buf][i] = __builtin_bit_cast(mf_t, t);
#endif
    }
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      if (MI + j < lo || MI + j >= hi || j >= NI_LIVE) continue;
#if B_FRTR
      bf[buf][j] = lds_frag_tr(lb, b_ft(lane, w, j, s, 0), b_ft(lane, w, j, s, 1));
#elif B_FRVEC
      bf[buf][j] = lds_frag(lb, b_fr(lane, w, j, s, 0));
#elif B_FRDW && B_FRDW_D
      {
        const IDX_T o0 = b_fd(lane, w, j, s, 0), o1 = b_fd(lane, w, j, s, 1);
        bf[buf][j] = lds_frag_dw(lb, o0, o0 + B_FRDW_D, o1, o1 + B_FRDW_D);
      }
#elif B_FRDW
      bf[buf][j] = lds_frag_dw(lb, b_fr(lane, w, j, s, 0), b_fr(lane, w, j, s, 2), b_fr(lane, w, j, s, 4),
                               b_fr(lane, w, j, s, 6));
#else
      e8_t t;
#pragma unroll
      for (int e = 0; e < 8; ++e) t[e] = lb[b_fr(lane, w, j, s, e)];
      bf[buf][j] = __builtin_bit_cast(mf_t, t);
#endif
    }
  };
  auto fload = [&](const elem_t* la, const elem_t* lb, int s, int buf) { fload_part(la, lb, s, buf, 0, MI + NI); };

  // Row r of the MFMAs of one substep with fragment set fb: every MFMA of a
  // row has the same first operand, A's fragment r.
#define MFMA_ROWS MI
  // The A operand of MFMA block row r.  With row pairs (A_FRZP) the
  // fragment registers of blocks 2m, 2m+1 hold the two 16-byte slots as read
  // (dwords: row 2r at k, k+1; row 2r+1 at k, k+1; then k+2, k+3), and the
  // operand is picked out here, when the MFMAs use it, so the register moves
  // never wait for the reads.
  auto a_op = [&](int r, int fb) -> mf_t {
#if A_FRZP
    const u4_t x0 = __builtin_bit_cast(u4_t, af[fb][r & ~1]), x1 = __builtin_bit_cast(u4_t, af[fb][r | 1]);
    const int p = r & 1;
    return __builtin_bit_cast(mf_t, (u4_t){x0[p], x0[p + 2], x1[p], x1[p + 2]});
#else
    return af[fb][r];
#endif
  };
  // Blocks past MI_LIVE / NI_LIVE hold no element of C in any tile: they
  // are neither read nor multiplied (their dead reads could otherwise share
  // registers with live values while in flight).
  auto mfma_row = [&](int r, int fb) {
    if (r >= MI_LIVE) return;
    const mf_t a = a_op(r, fb);
#pragma unroll
    for (int j = 0; j < NI_LIVE; ++j) acc[r][j] = MFMA(a, bf[fb][j], acc[r][j]);
  };
  auto mfma_all = [&](int fb) {
#pragma unroll
    for (int r = 0; r < MFMA_ROWS; ++r) mfma_row(r, fb);
  };

  // One K step on LDS stage kt&1.  `lbuf`: staging set receiving tile
  // kt+PREFETCH; `sbuf`: staging set holding tile kt+1, written to the other
  // LDS stage during the step.  The stage being written was last read in
  // step kt-1, whose closing barrier retired all of its readers.
  auto step = [&](IDX_T kt, int lbuf, int sbuf) {
    const int cur = kt & 1;
    if (kt + PREFETCH < KT) gload(kt + PREFETCH, lbuf);
    // Keep the loads at the top: the compiler would otherwise sink them to
    // their LDS stores.
    __builtin_amdgcn_sched_barrier(0);
    const elem_t* la = lds + cur * STAGE;
    const elem_t* lb = la + A_STAGE;
    fload(la, lb, 0, 0);
#pragma unroll
    for (int s = 0; s < BK / KB; ++s) {
      FRAG_WAIT();
      if (s + 1 < BK / KB) fload(la, lb, s + 1, (s + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);
      if (s == STORE_AT && kt + 1 < KT) sstore(cur ^ 1, sbuf);
      mfma_all(s & 1);
      if (s == STORE_AT) {
        // Spread the LDS stores between the MFMAs of this substep.
#pragma unroll
        for (int g = 0; g < A_NV * (A_SVEC ? A_VR : A_V) + B_NV * (B_SVEC ? B_VR : B_V); ++g) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
          __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // one LDS write
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
  };

#if DIRECT_LDS
  // Direct global-to-LDS copies: each lane's 16 bytes land at a wave-uniform
  // LDS base + 16 * lane, so load vector q = u*NT + tid fills LDS slot q; the
  // planner gave that lane the global address of the logical element the LDS
  // layout puts in slot q (the inverse of the LDS layout drives the copy).
  // NSTAGES LDS stages form a ring over the k-steps: the tile for step
  // g+NSTAGES is requested during step g, right after the barrier of its last
  // substep, into the stage step g has just finished reading.
  //
  // The grid is persistent when the launch makes it so (fewer workgroups than
  // output tiles): workgroup b computes the tiles whose schedule index is b,
  // b + G, b + 2G, ... (G = gridDim.x, every workgroup on the XCD that b is
  // dispatched to).  The ring runs on across tile boundaries: the last steps
  // of one tile request the first steps of the next, so the C stores of a
  // tile are issued while the next tile's operands are already on the way.
  const IDX_T wu = __builtin_amdgcn_readfirstlane(tid / 64u);
#if A_BUF || B_BUF
  // Range-checked buffer loads: an offset past the buffer's end (0xFFFFFFFF
  // for padding) writes zero to the LDS slot instead of reading memory.
  const __amdgpu_buffer_rsrc_t a_rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)A, (short)0, (int)A_BYTES, 0x00020000);
  const __amdgpu_buffer_rsrc_t b_rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)B, (short)0, (int)B_BYTES, 0x00020000);
#endif
  // One output tile: its coordinates and operand bases.
  struct Tile {
    IDX_T tm, tn;
    const elem_t* ab;
    const elem_t* bb;
  };
  auto tile_of = [&](IDX_T p) {
    Tile t;
    sched(p, &t.tm, &t.tn);
#if A_SEP
    t.ab = A + a_gt(t.tm);
#else
    t.ab = A;
#endif
#if B_SEP
    t.bb = B + b_gt(t.tn);
#else
    t.bb = B;
#endif
    return t;
  };
  // Copies [lo, hi) of step kt of tile t (A's A_NV vectors, then B's).
  auto dload_part = [&](const Tile& t, IDX_T kt, int stage, int lo, int hi) {
    elem_t* la = lds + stage * STAGE;
    elem_t* lb = la + A_STAGE;
#pragma unroll
    for (int u = 0; u < A_NV; ++u) {
      if (u < lo || u >= hi) continue;
#if A_SEP
      const elem_t* src = t.ab + a_gk(kt) + a_loc[u];
#else
      const elem_t* src = A + a_gf(t.tm, kt, tid, u);
#endif
      __attribute__((address_space(3))) void* dst = (__attribute__((address_space(3))) void*)(la + ((IDX_T)u * NT + wu * 64u) * 8u);
#if A_BUF
#if A_EDGE
      const unsigned off = a_ok(t.tm, kt, tid, u) ? (unsigned)((src - A) * 2) : 0xFFFFFFFFu;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(a_rsrc, dst, 16, off, 0, 0, 0);
#elif A_SEP
      // The lane's byte offset is fixed; the tile and k-step part is one
      // scalar offset, so a copy costs no vector arithmetic.
      (void)src;
      const unsigned soff = (unsigned)((t.ab - A) + a_gk(kt)) * 2u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(a_rsrc, dst, 16, a_loc[u] * 2u, soff, 0, 0);
#else
      __builtin_amdgcn_raw_ptr_buffer_load_lds(a_rsrc, dst, 16, (unsigned)((src - A) * 2), 0, 0, 0);
#endif
#else
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src, dst, 16, 0, 0);
#endif
    }
#pragma unroll
    for (int u = 0; u < B_NV; ++u) {
      if (A_NV + u < lo || A_NV + u >= hi) continue;
#if B_SEP
      const elem_t* src = t.bb + b_gk(kt) + b_loc[u];
#else
      const elem_t* src = B + b_gf(t.tn, kt, tid, u);
#endif
      __attribute__((address_space(3))) void* dst = (__attribute__((address_space(3))) void*)(lb + ((IDX_T)u * NT + wu * 64u) * 8u);
#if B_BUF
#if B_EDGE
      const unsigned off = b_ok(t.tn, kt, tid, u) ? (unsigned)((src - B) * 2) : 0xFFFFFFFFu;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(b_rsrc, dst, 16, off, 0, 0, 0);
#elif B_SEP
      (void)src;
      const unsigned soff = (unsigned)((t.bb - B) + b_gk(kt)) * 2u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(b_rsrc, dst, 16, b_loc[u] * 2u, soff, 0, 0);
#else
      __builtin_amdgcn_raw_ptr_buffer_load_lds(b_rsrc, dst, 16, (unsigned)((src - B) * 2), 0, 0, 0);
#endif
#else
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src, dst, 16, 0, 0);
#endif
    }
  };
  // s_waitcnt with only vmcnt constrained (expcnt and lgkmcnt at their maxima).
#define VMCNT_WAIT(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | ((((n) >> 4) & 3) << 14) | 0x70 | 0xF00)
  // Wait until at most `after` tiles of direct loads are still in flight.
  static_assert((NSTAGES - 1) * (A_NV + B_NV) <= 63, "vmcnt counts at most 63 loads");
  auto wait_tiles = [&](int after) {
    if (after <= 0) VMCNT_WAIT(0);
    else if (after == 1) VMCNT_WAIT(1 * (A_NV + B_NV));
#if NSTAGES > 2
    else if (after == 2) VMCNT_WAIT(2 * (A_NV + B_NV));
#endif
#if NSTAGES > 3
    else VMCNT_WAIT(3 * (A_NV + B_NV));  // (waits longer than needed beyond 3)
#endif
  };
  const IDX_T ntiles = (IDX_T)(GEMM_MT * GEMM_NT);
  IDX_T pid = blockIdx.x;
  Tile cur = tile_of(pid);
  // Every stage of the ring is filled up front; afterwards step g+NSTAGES is
  // requested as soon as the barrier of step g has retired the last reader of
  // its stage (a substep before step g+1 begins).  Every step requests one
  // step's copies (with fewer k-steps than stages, repeats of the tile's
  // steps), so the number in flight at each barrier is always the same.
#pragma unroll
  for (int p = 0; p < NSTAGES; ++p) dload_part(cur, (IDX_T)p % KT, p, 0, A_NV + B_NV);
  wait_tiles(NSTAGES - 1);
  __syncthreads();
  // Fragments are read FRAG_DIST substeps ahead of their MFMAs; the barrier
  // that hands over the LDS stages sits FRAG_DIST substeps before the end of
  // a step, so reads of the next stage can start there.
#pragma unroll
  for (int p = 0; p < FRAG_DIST; ++p) fload(lds, lds + A_STAGE, p, p % NFB);
  // One K step on LDS stage `cur_stage`; during it, step ck of tile `ct` is
  // requested into the same stage.  The body has no branch: a branch would
  // keep the scheduler from placing the copies and the fragment reads between
  // the MFMAs.
  auto kstep = [&](int cur_stage, const Tile& ct, IDX_T ck) {
    constexpr int S = BK / KB;
    const elem_t* la = lds + cur_stage * STAGE;
    const elem_t* na = lds + ((cur_stage + 1) % NSTAGES) * STAGE;
#pragma unroll
    for (int s = 0; s < S; ++s) {
      FRAG_WAIT_NEXT();
      if (s == S - FRAG_DIST) {
        // Every read of stage `cur_stage` has been issued and has completed
        // (the barrier waits for this wave's LDS reads).  Once the next step's
        // copies have landed (those requested after it may stay in flight)
        // and all waves are here, the stage is free for step g+NSTAGES and
        // the fragments of step g+1 can be read.
        wait_tiles(NSTAGES - 2);
        // This wave's reads of the stage must be complete before any wave
        // copies into it (the barrier alone does not wait for LDS reads).
        __builtin_amdgcn_s_waitcnt(0xC07F);
        __syncthreads();
        __builtin_amdgcn_sched_barrier(0);
      }
      // Reads for substep t of this step, or of the next one past the end.
      const int t = s + FRAG_DIST;
      const elem_t* ra = t < S ? la : na;
      const int ts = t < S ? t : t - S;
#if DMA_SPREAD
      if (s >= S - FRAG_DIST) {
        // The copies of step g+NSTAGES go out between the rows of MFMAs, a
        // share after each row, so the matrix pipe is never left idle while
        // the wave issues a burst of them; the fragment reads go out after
        // the first row, and the remaining rows cover their latency.
#pragma unroll
        for (int i = 0; i < MFMA_ROWS; ++i) {
          constexpr int R = DMA_ROWS;
          const int r = (s - (S - FRAG_DIST)) * MFMA_ROWS + i;
#if FRAG_SPREAD
          // Each row: its MFMAs with this row's share of the copies and of
          // the next fragments between them, one instruction after each MFMA.
          mfma_row(i, s % NFB);
          if (r < R) dload_part(ct, ck, cur_stage, r * (A_NV + B_NV) / R, (r + 1) * (A_NV + B_NV) / R);
          fload_part(ra, ra + A_STAGE, ts, ts % NFB, i * (MI + NI) / MI, (i + 1) * (MI + NI) / MI);
          // after MFMA g of the row: a copy (even g) or a fragment read (odd
          // g); with FRAG_SPREAD 3 the copy's LDS address (M0) is set one
          // MFMA ahead, so no wait state separates the two
#pragma unroll
          for (int g = 0; g < NI; ++g) {
            if (FRAG_SPREAD >= 3 && g % 2 == 0 && g / 2 < (A_NV + B_NV) / R)
              __builtin_amdgcn_sched_group_barrier(0x004, 1, 0);  // M0
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
            if (g % 2 == 0 && g / 2 < (A_NV + B_NV) / R) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
            if (g % 2 == 1 && g / 2 < (MI + NI) / MI) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
          __builtin_amdgcn_sched_barrier(0);
#else
          mfma_row(i, s % NFB);
          __builtin_amdgcn_sched_barrier(0);
          if (r < R) dload_part(ct, ck, cur_stage, r * (A_NV + B_NV) / R, (r + 1) * (A_NV + B_NV) / R);
          if (i == 0) fload(ra, ra + A_STAGE, ts, ts % NFB);
          __builtin_amdgcn_sched_barrier(0);
#endif
        }
        continue;
      }
#else
      if (s == S - FRAG_DIST) dload_part(ct, ck, cur_stage, 0, A_NV + B_NV);
#endif
#if FRAG_SPREAD >= 2
      // The next fragments go out one after each MFMA of the first rows, so
      // that the last is issued well before the substep ends (the substep
      // before the stage barrier waits for all of them).
      {
        // FR reads over the first ROWS rows (one per MFMA where the rows have
        // enough MFMAs; the rows present take them all otherwise).
        constexpr int FR = MI + NI;
        constexpr int ROWS = (FR + NI - 1) / NI < MFMA_ROWS ? (FR + NI - 1) / NI : MFMA_ROWS;
#pragma unroll
        for (int i = 0; i < MFMA_ROWS; ++i) {
          mfma_row(i, s % NFB);
          if (i < ROWS) {
            fload_part(ra, ra + A_STAGE, ts, ts % NFB, i * FR / ROWS, (i + 1) * FR / ROWS);
#pragma unroll
            for (int g = 0; g < NI; ++g) {
              __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
              __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      continue;
#endif
      mfma_all(s % NFB);
      // The reads are placed between these MFMAs, never ahead of them: with
      // direct loads in flight the only wait the compiler can place before an
      // MFMA is one for every outstanding LDS read, so a read issued before
      // this block would stall it.
      fload(ra, ra + A_STAGE, ts, ts % NFB);
#pragma unroll
      for (int g = 0; g < (FRAG_READS < MI * NI ? FRAG_READS : MI * NI); ++g) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
      }
      __builtin_amdgcn_sched_group_barrier(0x008, MI * NI, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, FRAG_READS, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // The stage of the current tile's step 0 (the ring advances KT steps per
  // tile).
  IDX_T stage0 = 0;
  // The k-loop's trip count is hidden from the compiler.  Unrolled in full
  // (K of two or three steps), the steps and the next tile's set-up become
  // one straight-line block whose register demand spilled, and the fragment
  // reads of the last step, dead there, shared registers with live values
  // while still in flight.
  IDX_T kt_end = KT;
  asm volatile("" : "+s"(kt_end));
  for (;;) {
    const IDX_T npid = pid + (IDX_T)gridDim.x;
    const bool has_next = PERSIST && npid < ntiles;
    // The last NSTAGES steps of a tile request the first steps of the next
    // one; the workgroup's last tile requests its own first steps again
    // (landing in stages nothing reads), which keeps every step alike.
    const Tile nxt = tile_of(has_next ? npid : pid);
    if constexpr (RING_UNROLL && KT % NSTAGES == 0) {
      // Every tile starts on stage 0: with the loop unrolled over the ring,
      // each step's stage is a constant and its fragment addresses are
      // loop-invariant registers (1.6% on the 8192^3 bf16 GEMM; plans with
      // two waves per SIMD lack the registers for them).
      // (a do-while: the compiler must see that a tile runs at least one
      // step, or on the path without steps it would reuse the registers of
      // fragment reads still in flight)
      IDX_T kt = 0;
      do {
#pragma unroll
        for (int p = 0; p < NSTAGES; ++p) {
          const bool own = kt + p + NSTAGES < KT;
          kstep(p, own ? cur : nxt, (kt + p + NSTAGES) % KT);
        }
        kt += NSTAGES;
      } while (kt < kt_end);
    } else {
      IDX_T kt = 0;
      do {
        const bool own = kt + NSTAGES < KT;
        kstep((int)((stage0 + kt) % NSTAGES), own ? cur : nxt, (kt + NSTAGES) % KT);
        ++kt;
      } while (kt < kt_end);
    }
    // After the workgroup's last tile the fragment reads issued by the last
    // step are dead, and the epilogue may reuse their registers: wait for
    // them first (between tiles they hold the next tile's fragments, which
    // stay live across the epilogue).
    if (!has_next) {
      FRAG_WAIT();
#if A_FRTR || B_FRTR
      // The trailing reads (substeps 0 .. FRAG_DIST-1 of a step that does
      // not exist) are dead to the compiler, which would hand their
      // registers to the epilogue as soon as the reads are issued: using
      // them here, after the wait, keeps them allocated until it.
#pragma unroll
      for (int t = 0; t < FRAG_DIST; ++t) {
#pragma unroll
        for (int i = 0; i < MI_LIVE; ++i)
          if (A_FRTR) asm volatile("" ::"v"(af[t % NFB][i]));
#pragma unroll
        for (int j = 0; j < NI_LIVE; ++j)
          if (B_FRTR) asm volatile("" ::"v"(bf[t % NFB][j]));
      }
#endif
    }
    store_c(cur.tm, cur.tn);
    if (!has_next) break;
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NI; ++j) acc[i][j] = (acc_t){};
    pid = npid;
    cur = nxt;
    stage0 = (stage0 + KT) % NSTAGES;
  }
  // The fragment reads and copies issued by the last step are not used; they
  // complete before the workgroup ends and before their registers are reused.
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_sched_barrier(0);
#elif (PREFETCH == 2 || ROLLING) && BK / KB >= 2
  // Register-staged pipeline.  With one wave per SIMD (the accumulators
  // fill the AGPRs) no other wave hides a stall, and with two the loads and
  // stores still cost less spread out: each step overlaps all of its memory
  // traffic with its MFMAs.  One staging set rolls through the tiles: during step t-1, in the
  // substeps before the last, each part of tile t is written from the set
  // to LDS stage t&1, and one substep later the same part of tile t+1 is
  // loaded into the freed registers (about a step ahead of its own LDS
  // write).  A barrier ahead of
  // the last substep publishes tile t, and that substep's MFMAs run under
  // the first fragment reads of step t.  Stage t&1 was last read in step
  // t-2, before that step's barrier.
  constexpr int S = BK / KB;
  constexpr int NL = A_NV + B_NV;  // load / store vectors per thread and tile
  auto pipe_step = [&](IDX_T kt) {
    const int cur = kt & 1;
    const elem_t* la = lds + cur * STAGE;
    const elem_t* lb = la + A_STAGE;
#pragma unroll
    for (int s = 0; s < S; ++s) {
      FRAG_WAIT();
      if (s == S - 1) {
        // this wave's stores of tile kt+1 are issued; once every wave's
        // have landed, stage (kt+1)&1 may be read
        __syncthreads();
        __builtin_amdgcn_sched_barrier(0);
      }
      mfma_all(s & 1);
      if (s + 1 < S) fload(la, lb, s + 1, (s + 1) & 1);
      else if (kt + 1 < KT) {
        const elem_t* na = lds + (cur ^ 1) * STAGE;
        fload(na, na + A_STAGE, 0, 0);
      }
      // Part s of tile kt+1 goes to LDS; part s-1, written one substep
      // earlier, is reloaded with tile kt+2 (reloading registers that an LDS
      // write still has to read would stall the wave until that write drains).
      if (s < S - 1 && kt + 1 < KT) sstore_part(cur ^ 1, 0, s * NL / (S - 1), (s + 1) * NL / (S - 1));
      if (s > 0 && kt + 2 < KT) gload_part(kt + 2, 0, (s - 1) * NL / (S - 1), s * NL / (S - 1));
      // one MFMA, then one of each kind of memory instruction, while they last
#pragma unroll
      for (int g = 0; g < MI * NI; ++g) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // LDS write
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // global load
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  gload(0, 0);
  sstore(0, 0);
  if (1 < KT) gload(1, 0);
  __syncthreads();
  fload(lds, lds + A_STAGE, 0, 0);
  for (IDX_T kt = 0; kt < KT; ++kt) pipe_step(kt);
#elif PREFETCH == 2
  gload(0, 0);
  if (1 < KT) gload(1, 1);
  sstore(0, 0);
  __syncthreads();
  for (IDX_T kt = 0; kt < KT; kt += 2) {
    step(kt, 0, 1);
    if (kt + 1 < KT) step(kt + 1, 1, 0);
  }
#else
  // Single staging set: the tile for step kt+1 is loaded at the top of step
  // kt and stored during it.
  gload(0, 0);
  sstore(0, 0);
  __syncthreads();
  for (IDX_T kt = 0; kt < KT; ++kt) {
    if (kt + 1 < KT) gload(kt + 1, 0);
    __builtin_amdgcn_sched_barrier(0);
    const int cur = kt & 1;
    const elem_t* la = lds + cur * STAGE;
    const elem_t* lb = la + A_STAGE;
    fload(la, lb, 0, 0);
#pragma unroll
    for (int s = 0; s < BK / KB; ++s) {
      FRAG_WAIT();
      if (s + 1 < BK / KB) fload(la, lb, s + 1, (s + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);
      if (s == STORE_AT && kt + 1 < KT) sstore(cur ^ 1, 0);
      mfma_all(s & 1);
      if (s == STORE_AT) {
#pragma unroll
        for (int g = 0; g < A_NV * (A_SVEC ? A_VR : A_V) + B_NV * (B_SVEC ? B_VR : B_V); ++g) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
  }
#endif
#if !DIRECT_LDS
  store_c(tm, tn);
#endif
}
