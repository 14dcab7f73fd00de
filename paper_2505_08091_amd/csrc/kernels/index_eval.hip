// Index-map evaluation kernels.  Generated code defines, before this text:
//   IDX_T, OUT_T, RANK, NPOINTS (u64 literal), PPT (outputs per 16-byte vector),
//   NT_STORE (1: streaming stores)
//   LEGO_FN IDX_T lego_map(IDX_T x)            logical flat index -> apply()
//   LEGO_FN void  lego_inv(IDX_T p, IDX_T* o)   physical index -> inv(), RANK outputs
// Outputs are written in point order, PPT consecutive points per thread so
// that every store is a whole 16-byte vector; the kernels are bound by the
// HBM write stream.  A grid-stride loop covers the points (normally one round:
// the grid covers every vector); the last partial group of points is written
// element by element.

// PPT (from the generated code): 16 / sizeof(OUT_T) outputs per 16-byte vector
typedef OUT_T ovec_t __attribute__((ext_vector_type(PPT)));
#if NT_STORE
#define IDX_ST(v, p) __builtin_nontemporal_store((v), (p))
#else
#define IDX_ST(v, p) (*(p) = (v))
#endif

#ifdef LEGO_HAVE_APPLY
extern "C" __global__ __launch_bounds__(256) void lego_apply_all(OUT_T* __restrict__ out) {
  const u64 stride = (u64)gridDim.x * 256u * PPT;
  for (u64 x0 = ((u64)blockIdx.x * 256u + threadIdx.x) * PPT; x0 < NPOINTS; x0 += stride) {
    if (x0 + PPT <= NPOINTS) {
      ovec_t v;
#pragma unroll
      for (int e = 0; e < PPT; ++e) v[e] = (OUT_T)lego_map((IDX_T)(x0 + e));
      IDX_ST(v, (ovec_t*)(out + x0));
    } else {
      for (u64 x = x0; x < NPOINTS; ++x) out[x] = (OUT_T)lego_map((IDX_T)x);
    }
  }
}
#endif

#ifdef LEGO_HAVE_INV
#define NOUT (NPOINTS * RANK)  // outputs: RANK coordinates per point
extern "C" __global__ __launch_bounds__(256) void lego_inv_all(OUT_T* __restrict__ out) {
  const u64 stride = (u64)gridDim.x * 256u * PPT;
#if PPT % RANK == 0
  // Each thread writes a run of PPT consecutive outputs (PPT / RANK whole
  // points), so the 64 lanes of a store cover one contiguous span.
  for (u64 f0 = ((u64)blockIdx.x * 256u + threadIdx.x) * PPT; f0 < NOUT; f0 += stride) {
    const u64 p0 = f0 / RANK;
    if (f0 + PPT <= NOUT) {
      ovec_t v;
#pragma unroll
      for (int e = 0; e < PPT / RANK; ++e) {
        IDX_T t[RANK];
        lego_inv((IDX_T)(p0 + e), t);
#pragma unroll
        for (int k = 0; k < RANK; ++k) v[e * RANK + k] = (OUT_T)t[k];
      }
      IDX_ST(v, (ovec_t*)(out + f0));
    } else {
      for (u64 p = p0; p < NPOINTS; ++p) {
        IDX_T t[RANK];
        lego_inv((IDX_T)p, t);
#pragma unroll
        for (int k = 0; k < RANK; ++k) out[p * RANK + k] = (OUT_T)t[k];
      }
    }
  }
#else
  // Runs would straddle points: one point per thread per round.
  for (u64 p = ((u64)blockIdx.x * 256u + threadIdx.x); p < NPOINTS; p += stride / PPT) {
    IDX_T t[RANK];
    lego_inv((IDX_T)p, t);
#pragma unroll
    for (int k = 0; k < RANK; ++k) out[p * RANK + k] = (OUT_T)t[k];
  }
#endif
}
#endif
