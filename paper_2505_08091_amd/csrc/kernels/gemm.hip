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
//   NWAVES NT KT     waves per workgroup, threads (64 * NWAVES), K / BK
//   IN_BF16          1: bf16 inputs, 0: fp16
//   A_NV A_V A_SEP A_SVEC A_FRVEC A_NVEC A_GUARD (and B_*): vectors per thread
//       per K step, elements per vector, additively separable global offset,
//       vector LDS store, vector fragment read, vectors per tile, and whether
//       the last round of vectors covers only part of the threads
//   C_SEP
//   sched(pid, &tm, &tn)
//   a_gt(tm) a_gk(kt) a_gl(tid, u)   or   a_gf(tm, kt, tid, u)
//   a_s(tid, u, e)                   LDS element offset of element e of load vector u
//   a_fr(lane, w, mi, s, e)          LDS element offset of fragment element e
//   (b_* likewise with tn)
//   c_t(tm, tn) c_l(lane, w, mi, ni, r)   or   c_f(tm, tn, lane, w, mi, ni, r)

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

extern "C" __global__ __launch_bounds__(NT) void lego_gemm(const elem_t* __restrict__ A, const elem_t* __restrict__ B,
                                                           float* __restrict__ C) {
  __shared__ __attribute__((aligned(16))) elem_t lds[2 * STAGE];
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

  av_t ra[A_NV];
  bv_t rb[B_NV];
  acc_t acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j) acc[i][j] = (acc_t){};

  auto gload = [&](IDX_T kt) {
#pragma unroll
    for (int u = 0; u < A_NV; ++u) {
      if (A_GUARD && (IDX_T)u * NT + tid >= A_NVEC) continue;
#if A_SEP
      ra[u] = *(const av_t*)(Ab + a_gk(kt) + a_loc[u]);
#else
      ra[u] = *(const av_t*)(A + a_gf(tm, kt, tid, u));
#endif
    }
#pragma unroll
    for (int u = 0; u < B_NV; ++u) {
      if (B_GUARD && (IDX_T)u * NT + tid >= B_NVEC) continue;
#if B_SEP
      rb[u] = *(const bv_t*)(Bb + b_gk(kt) + b_loc[u]);
#else
      rb[u] = *(const bv_t*)(B + b_gf(tn, kt, tid, u));
#endif
    }
  };
  auto sstore = [&](int stage) {
    elem_t* la = lds + stage * STAGE;
    elem_t* lb = la + A_STAGE;
#pragma unroll
    for (int u = 0; u < A_NV; ++u) {
      if (A_GUARD && (IDX_T)u * NT + tid >= A_NVEC) continue;
#if A_SVEC
      *(av_t*)(la + a_s(tid, u, 0)) = ra[u];
#else
#pragma unroll
      for (int e = 0; e < A_V; ++e) la[a_s(tid, u, e)] = ra[u][e];
#endif
    }
#pragma unroll
    for (int u = 0; u < B_NV; ++u) {
      if (B_GUARD && (IDX_T)u * NT + tid >= B_NVEC) continue;
#if B_SVEC
      *(bv_t*)(lb + b_s(tid, u, 0)) = rb[u];
#else
#pragma unroll
      for (int e = 0; e < B_V; ++e) lb[b_s(tid, u, e)] = rb[u][e];
#endif
    }
  };

  gload(0);
  sstore(0);
  __syncthreads();

  for (IDX_T kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT) gload(kt + 1);
    const elem_t* la = lds + cur * STAGE;
    const elem_t* lb = la + A_STAGE;
#pragma unroll
    for (int s = 0; s < BK / KB; ++s) {
      mf_t af[MI], bf[NI];
#pragma unroll
      for (int i = 0; i < MI; ++i) {
#if A_FRVEC
        af[i] = lds_frag(la, a_fr(lane, w, i, s, 0));
#else
        e8_t t;
#pragma unroll
        for (int e = 0; e < 8; ++e) t[e] = la[a_fr(lane, w, i, s, e)];
        af[i] = __builtin_bit_cast(mf_t, t);
#endif
      }
#pragma unroll
      for (int j = 0; j < NI; ++j) {
#if B_FRVEC
        bf[j] = lds_frag(lb, b_fr(lane, w, j, s, 0));
#else
        e8_t t;
#pragma unroll
        for (int e = 0; e < 8; ++e) t[e] = lb[b_fr(lane, w, j, s, e)];
        bf[j] = __builtin_bit_cast(mf_t, t);
#endif
      }
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NI; ++j) acc[i][j] = MFMA(af[i], bf[j], acc[i][j]);
    }
    if (kt + 1 < KT) sstore(cur ^ 1);
    __syncthreads();
  }

#if C_SEP
  float* __restrict__ Cb = C + c_t(tm, tn);
#endif
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j)
#pragma unroll
      for (int r = 0; r < NREG; ++r) {
#if C_SEP
        __builtin_nontemporal_store(acc[i][j][r], Cb + c_l(lane, w, i, j, r));
#else
        __builtin_nontemporal_store(acc[i][j][r], C + c_f(tm, tn, lane, w, i, j, r));
#endif
      }
}
