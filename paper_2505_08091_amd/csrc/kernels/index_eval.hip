// Index-map evaluation kernels.  Generated code defines, before this text:
//   IDX_T, OUT_T, RANK, NPOINTS (u64 literal)
//   LEGO_FN IDX_T lego_map(IDX_T x)            logical flat index -> apply()
//   LEGO_FN void  lego_inv(IDX_T p, IDX_T* o)   physical index -> inv(), RANK outputs
// Each thread handles points in a grid-stride loop; outputs are written in
// point order, so stores are fully coalesced (the kernels are bound by the
// HBM write stream).

#ifdef LEGO_HAVE_APPLY
extern "C" __global__ __launch_bounds__(256) void lego_apply_all(OUT_T* __restrict__ out) {
  const u64 stride = (u64)gridDim.x * 256u;
  for (u64 x = (u64)blockIdx.x * 256u + threadIdx.x; x < NPOINTS; x += stride)
    out[x] = (OUT_T)lego_map((IDX_T)x);
}
#endif

#ifdef LEGO_HAVE_INV
extern "C" __global__ __launch_bounds__(256) void lego_inv_all(OUT_T* __restrict__ out) {
  const u64 stride = (u64)gridDim.x * 256u;
  for (u64 p = (u64)blockIdx.x * 256u + threadIdx.x; p < NPOINTS; p += stride) {
    IDX_T o[RANK];
    lego_inv((IDX_T)p, o);
#pragma unroll
    for (int k = 0; k < RANK; ++k) out[p * RANK + k] = (OUT_T)o[k];
  }
}
#endif
