// Backward pass of Sparse Reference Attention on gfx950.
//
// The gradient of masked softmax attention (the textbook one; the paper trains through SRA
// in its personality fine-tuning stage, §3.3): with P = softmax of the scaled logits over
// the visible keys, D = rowsum(dO * O),
//     dV = P^T dO,   dP = dO V^T,   dS = P * (dP - D),   dQ = scale dS K,   dK = scale dS^T Q.
// Three kernels, all deterministic (no atomics):
//   delta : -D and the log-sum-exp in log2 units for every query row (HBM bound); the other
//           two kernels fetch both per row and use them without further arithmetic.
//   dq    : query-major, in sra_dq.hip.
//   dkv   : key-major, in sra_dkv.hip.
// P is recomputed from the forward's log-sum-exp. Spans' ragged ends, and in dK/dV the keys of
// a tile outside a span's key range, are the only masks.
#include "sra_kernels.h"
#include "sra_tiles.h"

namespace sra {

namespace {
constexpr float kLog2e = 1.44269504088896340736f;
}

// --------------------------------------------------------------------------- delta
template <int D>
__global__ void __launch_bounds__(kThreads) sra_delta_kernel(DeltaArgs a, int s) {
  constexpr int TPR = D / 8;                  // threads per (row, head)
  constexpr int RPB = kThreads / TPR;         // (row, head) pairs per block
  const int64_t pair = int64_t(blockIdx.x) * RPB + threadIdx.x / TPR;
  const int64_t total = int64_t(a.rows[s]) * a.heads;
  const int sub = threadIdx.x % TPR;
  float acc = 0.f;
  if (pair < total) {
    const int64_t row = pair / a.heads;
    const int h = int(pair % a.heads);
    const int64_t off = (row * a.heads + h) * D + sub * 8;
    const bf16x8 x = *reinterpret_cast<const bf16x8*>(a.o[s] + off);
    const bf16x8 y = *reinterpret_cast<const bf16x8*>(a.dout[s] + off);
#pragma unroll
    for (int j = 0; j < 8; ++j) acc = fmaf(float(x[j]), float(y[j]), acc);
  }
#pragma unroll
  for (int w = 1; w < TPR; w <<= 1) acc += __shfl_xor(acc, w, TPR);
  if (pair < total && sub == 0) {
    const int64_t row = pair / a.heads;
    const int h = int(pair % a.heads);
    const int64_t i = int64_t(h) * a.rows[s] + row;
    a.ndelta[s][i] = -acc;
    a.lse2[s][i] = a.lse[s][i] * kLog2e;
  }
}

hipError_t launch_delta(const DeltaArgs& a, int head_dim, hipStream_t stream) {
  for (int s = 0; s < 2; ++s) {
    const int64_t total = int64_t(a.rows[s]) * a.heads;
    if (total == 0) continue;
    const int rpb = kThreads / (head_dim / 8);
    const unsigned blocks = unsigned((total + rpb - 1) / rpb);
    if (head_dim == 128)
      hipLaunchKernelGGL(sra_delta_kernel<128>, dim3(blocks), dim3(kThreads), 0, stream, a, s);
    else
      hipLaunchKernelGGL(sra_delta_kernel<64>, dim3(blocks), dim3(kThreads), 0, stream, a, s);
  }
  return hipGetLastError();
}

// --------------------------------------------------------------------------- fill
// Rows of invalid reference frames: outputs/gradients 0, log-sum-exp -inf.
__global__ void __launch_bounds__(kThreads) sra_fill_kernel(FillArgs a) {
  const FillRange r = a.ranges[blockIdx.x];
  const int64_t row_elems = int64_t(a.heads) * a.head_dim;
  const int64_t chunks = int64_t(r.len) * row_elems / 8;
  const int64_t base = int64_t(r.start) * row_elems;
  const int64_t stride = int64_t(gridDim.y) * blockDim.x;
  for (int64_t u = int64_t(blockIdx.y) * blockDim.x + threadIdx.x; u < chunks; u += stride) {
#pragma unroll
    for (int j = 0; j < 3; ++j)
      if (a.t[j]) *reinterpret_cast<uint4*>(a.t[j] + base + u * 8) = uint4{0, 0, 0, 0};
  }
  if (a.lse) {
    const int64_t n = int64_t(a.heads) * r.len;
    for (int64_t u = int64_t(blockIdx.y) * blockDim.x + threadIdx.x; u < n; u += stride) {
      const int64_t hh = u / r.len, i = u % r.len;
      a.lse[hh * a.lse_rows + r.start + i] = -INFINITY;
    }
  }
}

hipError_t launch_fill(const FillArgs& a, hipStream_t stream) {
  if (a.n_ranges <= 0) return hipSuccess;
  hipLaunchKernelGGL(sra_fill_kernel, dim3(a.n_ranges, 64), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace sra
