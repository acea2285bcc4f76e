// Row gather and scatter between the packed reference stream and its compacted form (the
// valid reference tokens back to back), used when a token mask splits reference frames into
// short runs. Plain HBM-bound copies: one workgroup per destination row, 16-byte accesses.
#include "sra_kernels.h"

namespace sra {

// dst[t][c] = src[t][index[c]] for every tensor t (whole rows of heads * D elements), and
// lse_dst[h][c] = lse_src[h][index[c]].
__global__ void __launch_bounds__(kThreads) sra_gather_kernel(GatherArgs a) {
  const int64_t c = blockIdx.x;
  const int64_t r = a.index[c];
  const int chunks = a.row_elems / 8;
#pragma unroll
  for (int t = 0; t < kGatherMax; ++t) {
    if (!a.src[t]) continue;
    const uint4* s = reinterpret_cast<const uint4*>(a.src[t] + r * a.src_stride[t]);
    uint4* d = reinterpret_cast<uint4*>(a.dst[t] + c * a.row_elems);
    for (int u = threadIdx.x; u < chunks; u += blockDim.x) d[u] = s[u];
  }
  if (a.lse_src)
    for (int h = threadIdx.x; h < a.heads; h += blockDim.x)
      a.lse_dst[int64_t(h) * a.rows + c] = a.lse_src[int64_t(h) * a.lse_src_rows + r];
}

// dst[t][r] = src[t][index[r]], or zeros where index[r] < 0 (invalid tokens); the same for
// the log-sum-exp rows, with -inf for invalid tokens.
__global__ void __launch_bounds__(kThreads) sra_scatter_kernel(ScatterArgs a) {
  const int64_t r = blockIdx.x;
  const int64_t c = a.index[r];
  const int chunks = a.row_elems / 8;
#pragma unroll
  for (int t = 0; t < kScatterMax; ++t) {
    if (!a.dst[t]) continue;
    uint4* d = reinterpret_cast<uint4*>(a.dst[t] + r * a.row_elems);
    if (c >= 0) {
      const uint4* s = reinterpret_cast<const uint4*>(a.src[t] + c * a.row_elems);
      for (int u = threadIdx.x; u < chunks; u += blockDim.x) d[u] = s[u];
    } else {
      for (int u = threadIdx.x; u < chunks; u += blockDim.x) d[u] = uint4{0, 0, 0, 0};
    }
  }
  if (a.lse_dst)
    for (int h = threadIdx.x; h < a.heads; h += blockDim.x)
      a.lse_dst[int64_t(h) * a.rows + r] = c >= 0 ? a.lse_src[int64_t(h) * a.lse_src_rows + c] : -INFINITY;
}

hipError_t launch_gather(const GatherArgs& a, hipStream_t stream) {
  if (a.rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(sra_gather_kernel, dim3(a.rows), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_scatter(const ScatterArgs& a, hipStream_t stream) {
  if (a.rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(sra_scatter_kernel, dim3(a.rows), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace sra
