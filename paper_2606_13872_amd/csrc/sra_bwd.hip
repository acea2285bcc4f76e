// Backward pass of Sparse Reference Attention on gfx950.
//
// The gradient of masked softmax attention (the textbook one; the paper trains through SRA
// in its personality fine-tuning stage, §3.3): with P = softmax of the scaled logits over
// the visible keys, D = rowsum(dO * O),
//     dV = P^T dO,   dP = dO V^T,   dS = P * (dP - D),   dQ = scale dS K,   dK = scale dS^T Q.
// Three kernels, all deterministic (no atomics):
//   delta : -D and the log-sum-exp in log2 units for every query row (HBM bound); the other
//           two kernels fetch both per row and use them without further arithmetic.
//   dq    : query-major, like the forward: S^T = K Q^T, dP^T = V dO^T, dQ^T += K^T dS^T.
//   dkv   : key-major, in sra_dkv.hip.
// P is recomputed from the forward's log-sum-exp. Spans' ragged ends are the only masks.
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

// --------------------------------------------------------------------------- dq
namespace {
constexpr int kDqWaves = kDqQueryTile / 32;
constexpr int kDqBufs = 4;
}

template <int D>
struct DqState {
  bf16x8 qf[D / 16];    // Q^T B fragments (lane = query)
  bf16x8 df[D / 16];    // dO^T B fragments (lane = query)
  floatx16 dq[D / 32];  // dQ^T accumulators, 32 head dims each
  float lse2, ndlt;     // the row's log-sum-exp (log2 units) and -rowsum(dO * O)
};

// One 32-key step of dQ for the wave's 32 query rows (S^T, dP^T with lanes = queries).
template <int D, bool kMask>
__device__ __forceinline__ void dq_step(DqState<D>& st, const __bf16* kt, const __bf16* vt, int nvalid,
                                        float sl2) {
  constexpr int NC = D / 16, ND = D / 32, RK = kBothPadRS<D>, RV = kRowPadRS<D>;
  const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
  floatx16 s = floatx16{}, dp = floatx16{};
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const bf16x8 ka = *reinterpret_cast<const bf16x8*>(kt + l32 * RK + c * 16 + half * 8);
    const bf16x8 va = *reinterpret_cast<const bf16x8*>(vt + l32 * RV + c * 16 + half * 8);
    s = mfma32(ka, st.qf[c], s);
    dp = mfma32(va, st.df[c], dp);
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    float p = fast_exp2(fmaf(s[i], sl2, -st.lse2));
    if constexpr (kMask) p = (8 * (i >> 2) + 4 * half + (i & 3)) < nvalid ? p : 0.f;
    s[i] = p * (dp[i] + st.ndlt);
  }
  // dQ^T += K^T dS^T ; K^T fragments through the transpose read
  const int tcol = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const int trow = 4 * half + ((lane & 15) >> 2);
#pragma unroll
  for (int c2 = 0; c2 < 2; ++c2) {
    const bf16x8 dsf = to_bf16x8(s, 8 * c2);
    const int r0 = 16 * c2 + trow;
#pragma unroll
    for (int db = 0; db < ND; ++db) {
      const bf16x8 kta = cat8(lds_read_tr(kt + r0 * RK + db * 32 + tcol),
                              lds_read_tr(kt + (r0 + 8) * RK + db * 32 + tcol));
      st.dq[db] = mfma32(kta, dsf, st.dq[db]);
    }
  }
}

template <int D>
__global__ void __launch_bounds__(kDqWaves * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
sra_dq_kernel(BwdArgs a) {
  constexpr int NC = D / 16, ND = D / 32, BK = kDqKeyStep, RK = kBothPadRS<D>, RV = kRowPadRS<D>;
  // K is read both as row fragments and through the transpose read, from one copy at D + 24
  // (measured faster here than the permuted-row layout or a second copy). Key tiles
  // rotate through kDqBufs buffers, are loaded two steps ahead, and the workgroup meets at a
  // barrier after every second step (as in the dK/dV kernel).
  constexpr int NB = kDqBufs;
  __shared__ __attribute__((aligned(1024))) __bf16 ks[NB][PaddedTile<D, BK, RK>::kElems];
  __shared__ __attribute__((aligned(1024))) __bf16 vs[NB][PaddedTile<D, BK, RV>::kElems];

  const WorkItem it = a.items[blockIdx.x];
  if (it.stream < 0) return;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int half = lane >> 5, l32 = lane & 31;
  const int h = it.head, s = it.stream;
  const bool active = wave * 32 < it.len;
  const float sl2 = a.scale_log2;

  DqState<D> st;
  const int r = wave * 32 + l32;
  {
    const int rr = it.start + min(r, it.len - 1);
    const __bf16* qs = a.q[s] + int64_t(rr) * a.in_stride[s] + h * D + half * 8;
    const __bf16* ds = a.dout[s] + int64_t(rr) * (int64_t(a.heads) * D) + h * D + half * 8;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const bf16x8 x = *reinterpret_cast<const bf16x8*>(qs + c * 16);
      const bf16x8 y = *reinterpret_cast<const bf16x8*>(ds + c * 16);
      st.qf[c] = (r < it.len) ? x : bf16x8{};
      st.df[c] = (r < it.len) ? y : bf16x8{};
    }
#pragma unroll
    for (int db = 0; db < ND; ++db) st.dq[db] = floatx16{};
    st.lse2 = a.lse2[s][int64_t(h) * a.rows[s] + rr];
    st.ndlt = a.ndelta[s][int64_t(h) * a.rows[s] + rr];
  }

  const Span* sp = a.spans + it.span_off;
  const int T = count_steps(sp, it.span_cnt, BK);
  SpanCursor ld;
  ld.init(sp, it.span_cnt);
  TileLoader<D, BK, RK, kDqWaves> kl[2];
  TileLoader<D, BK, RV, kDqWaves> vl[2];
#pragma unroll
  for (int ss = 0; ss < 2; ++ss) {
    kl[ss].init(a.in_stride[ss], h, wave);
    vl[ss].init(a.in_stride[ss], h, wave);
  }
  auto issue = [&](int b) {
    const int ss = ld.stream();
    if (ld.off + BK <= ld.len()) {
      const int64_t row0 = int64_t(ld.start() + ld.off) * a.in_stride[ss];
      if (ss == 0) {
        kl[0].issue(ks[b], a.k[0] + row0, wave);
        vl[0].issue(vs[b], a.v[0] + row0, wave);
      } else {
        kl[1].issue(ks[b], a.k[1] + row0, wave);
        vl[1].issue(vs[b], a.v[1] + row0, wave);
      }
    } else {
      tile_load_lds<D, BK, RK, kDqWaves>(ks[b], a.k[ss], a.in_stride[ss], h, ld.start(), ld.len(), ld.off, wave);
      tile_load_lds<D, BK, RV, kDqWaves>(vs[b], a.v[ss], a.in_stride[ss], h, ld.start(), ld.len(), ld.off, wave);
    }
    ld.advance(BK);
  };

  issue(0);
  if (T > 1) issue(1);
  wait_vmem();
  __syncthreads();
  // Step t reads buffer t % NB and loads step t + 2 into buffer (t + 2) % NB. That buffer's
  // last reader, step t - 2, finished before the barrier ending step t - 2 or t - 1
  // (whichever is odd); the tiles of step t landed before that same barrier.
  int t = 0;
  for (int si = 0; si < it.span_cnt; ++si) {
    const int len = __builtin_amdgcn_readfirstlane(sp[si].len);
    const int full = len / BK;
    for (int j = 0; j < full; ++j, ++t) {
      if (t + 2 < T) issue((t + 2) % NB);
      if (active) dq_step<D, false>(st, ks[t % NB], vs[t % NB], BK, sl2);
      if (t & 1) {
        wait_vmem();
        __syncthreads();
      }
    }
    if (len % BK) {
      if (t + 2 < T) issue((t + 2) % NB);
      if (active) dq_step<D, true>(st, ks[t % NB], vs[t % NB], len % BK, sl2);
      if (t & 1) {
        wait_vmem();
        __syncthreads();
      }
      ++t;
    }
  }

  if (!active || r >= it.len) return;
  __bf16* orow = a.dq[s] + int64_t(it.start + r) * (int64_t(a.heads) * D) + h * D;
#pragma unroll
  for (int db = 0; db < ND; ++db)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 w;
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = (__bf16)(st.dq[db][4 * g + e] * a.scale);
      *reinterpret_cast<bf16x4*>(orow + db * 32 + 8 * g + 4 * half) = w;
    }
}

hipError_t launch_dq(const BwdArgs& a, int n_items, int head_dim, hipStream_t stream) {
  if (n_items <= 0) return hipSuccess;
  if (head_dim == 128)
    hipLaunchKernelGGL(sra_dq_kernel<128>, dim3(n_items), dim3(kDqWaves * 64), 0, stream, a);
  else
    hipLaunchKernelGGL(sra_dq_kernel<64>, dim3(n_items), dim3(kDqWaves * 64), 0, stream, a);
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
