// Backward pass of Sparse Reference Attention on gfx950.
//
// The gradient of masked softmax attention (the textbook one; the paper trains through SRA
// in its personality fine-tuning stage, §3.3): with P = softmax of the scaled logits over
// the visible keys, D = rowsum(dO * O),
//     dV = P^T dO,   dP = dO V^T,   dS = P * (dP - D),   dQ = scale dS K,   dK = scale dS^T Q.
// Three kernels, all deterministic (no atomics):
//   delta : D for every query row (HBM bound).
//   dq    : query-major, like the forward: S^T = K Q^T, dP^T = V dO^T, dQ^T += K^T dS^T.
//   dkv   : key-major: each wave keeps 32 keys' K and V in VGPRs and streams the query rows
//           that see those keys (gen keys: the gen queries of the sample; ref keys: the gen
//           queries plus the ref queries of the key's group):
//             S = Q K^T, dP = dO V^T, dV^T += dO^T P, dK^T += Q^T dS.
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
    a.delta[s][int64_t(h) * a.rows[s] + row] = acc;
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
template <int D>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
sra_dq_kernel(BwdArgs a) {
  constexpr int NC = D / 16, ND = D / 32, BK = kDqKeyStep;
  __shared__ __attribute__((aligned(16))) __bf16 ks[2][BK * D];
  __shared__ __attribute__((aligned(16))) __bf16 vs[2][BK * D];

  const WorkItem it = a.items[blockIdx.x];
  if (it.stream < 0) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const int h = it.head, s = it.stream;
  const int wrow0 = wave * 64;
  const bool active = wrow0 < it.len;
  const float sl2 = a.scale_log2;

  bf16x8 qf[2][NC], df[2][NC];
  float lse2[2], dlt[2];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int r = wrow0 + qb * 32 + l32;
    const int rr = it.start + min(r, it.len - 1);
    const __bf16* qs = a.q[s] + int64_t(rr) * a.in_stride[s] + h * D + half * 8;
    const __bf16* ds = a.dout[s] + int64_t(rr) * (int64_t(a.heads) * D) + h * D + half * 8;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const bf16x8 x = *reinterpret_cast<const bf16x8*>(qs + c * 16);
      const bf16x8 y = *reinterpret_cast<const bf16x8*>(ds + c * 16);
      qf[qb][c] = (r < it.len) ? x : bf16x8{};
      df[qb][c] = (r < it.len) ? y : bf16x8{};
    }
    lse2[qb] = a.lse[s][int64_t(h) * a.rows[s] + rr] * kLog2e;
    dlt[qb] = a.delta[s][int64_t(h) * a.rows[s] + rr];
  }

  floatx16 dq[2][ND];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int db = 0; db < ND; ++db) dq[qb][db] = floatx16{};

  const Span* sp = a.spans + it.span_off;
  const int T = count_steps(sp, it.span_cnt, BK);
  SpanCursor ld, cp;
  ld.init(sp, it.span_cnt);
  cp.init(sp, it.span_cnt);
  TileRegs<D, BK> kr, vr;
  tile_load<D, BK>(kr, a.k[ld.stream()], a.in_stride[ld.stream()], h, ld.start(), ld.len(), ld.off);
  tile_load<D, BK>(vr, a.v[ld.stream()], a.in_stride[ld.stream()], h, ld.start(), ld.len(), ld.off);
  ld.advance(BK);
  tile_store<D, BK>(kr, ks[0]);
  tile_store<D, BK>(vr, vs[0]);
  __syncthreads();
  if (T > 1) {
    tile_load<D, BK>(kr, a.k[ld.stream()], a.in_stride[ld.stream()], h, ld.start(), ld.len(), ld.off);
    tile_load<D, BK>(vr, a.v[ld.stream()], a.in_stride[ld.stream()], h, ld.start(), ld.len(), ld.off);
    ld.advance(BK);
  }
  const int tcol = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const int trow = 4 * half + ((lane & 15) >> 2);

  for (int t = 0; t < T; ++t) {
    const int buf = t & 1;
    const int nvalid = min(BK, cp.len() - cp.off);
    if (active) {
      const __bf16* kt = ks[buf];
      const __bf16* vt = vs[buf];
      floatx16 st[2], dpt[2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        st[qb] = floatx16{};
        dpt[qb] = floatx16{};
      }
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const bf16x8 ka = *reinterpret_cast<const bf16x8*>(kt + tile_off<D>(l32, c * 16 + half * 8));
        const bf16x8 va = *reinterpret_cast<const bf16x8*>(vt + tile_off<D>(l32, c * 16 + half * 8));
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
          st[qb] = mfma32(ka, qf[qb][c], st[qb]);
          dpt[qb] = mfma32(va, df[qb][c], dpt[qb]);
        }
      }
      bf16x8 dsf[2][2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = 8 * (i >> 2) + 4 * half + (i & 3);
          float p = fast_exp2(fmaf(st[qb][i], sl2, -lse2[qb]));
          p = key < nvalid ? p : 0.f;
          st[qb][i] = p * (dpt[qb][i] - dlt[qb]);
        }
        dsf[qb][0] = to_bf16x8(st[qb], 0);
        dsf[qb][1] = to_bf16x8(st[qb], 8);
      }
      // dQ^T += K^T dS^T ; K^T fragments through the transpose read
#pragma unroll
      for (int db = 0; db < ND; ++db)
#pragma unroll
        for (int c2 = 0; c2 < 2; ++c2) {
          const int r0 = 16 * c2 + trow;
          const bf16x8 kta = cat8(lds_read_tr(kt + tile_off<D>(r0, db * 32 + tcol)),
                                  lds_read_tr(kt + tile_off<D>(r0 + 8, db * 32 + tcol)));
#pragma unroll
          for (int qb = 0; qb < 2; ++qb) dq[qb][db] = mfma32(kta, dsf[qb][c2], dq[qb][db]);
        }
    }
    cp.advance(BK);
    if (t + 1 < T) {
      tile_store<D, BK>(kr, ks[buf ^ 1]);
      tile_store<D, BK>(vr, vs[buf ^ 1]);
    }
    __syncthreads();
    if (t + 2 < T) {
      tile_load<D, BK>(kr, a.k[ld.stream()], a.in_stride[ld.stream()], h, ld.start(), ld.len(), ld.off);
      tile_load<D, BK>(vr, a.v[ld.stream()], a.in_stride[ld.stream()], h, ld.start(), ld.len(), ld.off);
      ld.advance(BK);
    }
  }

  if (!active) return;
  const int64_t ostride = int64_t(a.heads) * D;
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int r = wrow0 + qb * 32 + l32;
    if (r >= it.len) continue;
    __bf16* orow = a.dq[s] + int64_t(it.start + r) * ostride + h * D;
#pragma unroll
    for (int db = 0; db < ND; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = (__bf16)(dq[qb][db][4 * g + e] * a.scale);
        *reinterpret_cast<bf16x4*>(orow + db * 32 + 8 * g + 4 * half) = w;
      }
  }
}

hipError_t launch_dq(const BwdArgs& a, int n_items, int head_dim, hipStream_t stream) {
  if (n_items <= 0) return hipSuccess;
  if (head_dim == 128)
    hipLaunchKernelGGL(sra_dq_kernel<128>, dim3(n_items), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(sra_dq_kernel<64>, dim3(n_items), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

// --------------------------------------------------------------------------- dkv
template <int D>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
sra_dkv_kernel(BwdArgs a) {
  constexpr int NC = D / 16, ND = D / 32, BQ = kDkvQueryStep;
  __shared__ __attribute__((aligned(16))) __bf16 qs[2][BQ * D];
  __shared__ __attribute__((aligned(16))) __bf16 dos[2][BQ * D];
  __shared__ __attribute__((aligned(16))) float lse_s[2][BQ];
  __shared__ __attribute__((aligned(16))) float dlt_s[2][BQ];

  const WorkItem it = a.items[blockIdx.x];
  if (it.stream < 0) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const int h = it.head, s = it.stream;
  const int wkey0 = wave * 32;
  const bool active = wkey0 < it.len;
  const float sl2 = a.scale_log2;

  // K and V as MFMA B fragments: lane holds key l32 and 8 consecutive head dims.
  bf16x8 kf[NC], vf[NC];
  {
    const int r = wkey0 + l32;
    const int rr = it.start + min(r, it.len - 1);
    const __bf16* kp = a.k[s] + int64_t(rr) * a.in_stride[s] + h * D + half * 8;
    const __bf16* vp = a.v[s] + int64_t(rr) * a.in_stride[s] + h * D + half * 8;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const bf16x8 x = *reinterpret_cast<const bf16x8*>(kp + c * 16);
      const bf16x8 y = *reinterpret_cast<const bf16x8*>(vp + c * 16);
      kf[c] = (r < it.len) ? x : bf16x8{};
      vf[c] = (r < it.len) ? y : bf16x8{};
    }
  }
  floatx16 dk[ND], dv[ND];
#pragma unroll
  for (int db = 0; db < ND; ++db) {
    dk[db] = floatx16{};
    dv[db] = floatx16{};
  }

  const Span* sp = a.spans + it.span_off;
  const int T = count_steps(sp, it.span_cnt, BQ);
  SpanCursor ld, cp;
  ld.init(sp, it.span_cnt);
  cp.init(sp, it.span_cnt);
  TileRegs<D, BQ> qr, dr;
  float lr = 0.f, drr = 0.f;  // threads < BQ stage one row's LSE (log2 units) and delta

  auto load_step = [&]() {
    const int ss = ld.stream();
    tile_load<D, BQ>(qr, a.q[ss], a.in_stride[ss], h, ld.start(), ld.len(), ld.off);
    tile_load<D, BQ>(dr, a.dout[ss], int64_t(a.heads) * D, h, ld.start(), ld.len(), ld.off);
    if (threadIdx.x < BQ) {
      const int rr = ld.start() + min(ld.off + int(threadIdx.x), ld.len() - 1);
      lr = a.lse[ss][int64_t(h) * a.rows[ss] + rr] * kLog2e;
      drr = a.delta[ss][int64_t(h) * a.rows[ss] + rr];
    }
    ld.advance(BQ);
  };
  auto store_step = [&](int b) {
    tile_store<D, BQ>(qr, qs[b]);
    tile_store<D, BQ>(dr, dos[b]);
    if (threadIdx.x < BQ) {
      lse_s[b][threadIdx.x] = lr;
      dlt_s[b][threadIdx.x] = drr;
    }
  };

  load_step();
  store_step(0);
  __syncthreads();
  if (T > 1) load_step();
  const int tcol = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const int trow = 4 * half + ((lane & 15) >> 2);

  for (int t = 0; t < T; ++t) {
    const int buf = t & 1;
    const int nvalid = min(BQ, cp.len() - cp.off);
    if (active) {
      const __bf16* qt = qs[buf];
      const __bf16* dt = dos[buf];
      floatx16 st[2], dp[2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        st[qb] = floatx16{};
        dp[qb] = floatx16{};
      }
      // S = Q K^T and dP = dO V^T (rows = queries, lanes = keys)
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
          const bf16x8 qa = *reinterpret_cast<const bf16x8*>(qt + tile_off<D>(qb * 32 + l32, c * 16 + half * 8));
          const bf16x8 da = *reinterpret_cast<const bf16x8*>(dt + tile_off<D>(qb * 32 + l32, c * 16 + half * 8));
          st[qb] = mfma32(qa, kf[c], st[qb]);
          dp[qb] = mfma32(da, vf[c], dp[qb]);
        }
      bf16x8 pb[2][2], sb[2][2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int q0 = qb * 32 + 8 * g + 4 * half;  // 4 consecutive query rows
          const floatx4 l4 = *reinterpret_cast<const floatx4*>(&lse_s[buf][q0]);
          const floatx4 d4 = *reinterpret_cast<const floatx4*>(&dlt_s[buf][q0]);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int i = 4 * g + e;
            float p = fast_exp2(fmaf(st[qb][i], sl2, -l4[e]));
            p = (q0 + e) < nvalid ? p : 0.f;
            st[qb][i] = p;
            dp[qb][i] = p * (dp[qb][i] - d4[e]);
          }
        }
        pb[qb][0] = to_bf16x8(st[qb], 0);
        pb[qb][1] = to_bf16x8(st[qb], 8);
        sb[qb][0] = to_bf16x8(dp[qb], 0);
        sb[qb][1] = to_bf16x8(dp[qb], 8);
      }
      // dV^T += dO^T P and dK^T += Q^T dS ; dO^T and Q^T fragments via the transpose read
#pragma unroll
      for (int db = 0; db < ND; ++db)
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
          for (int c2 = 0; c2 < 2; ++c2) {
            const int r0 = qb * 32 + 16 * c2 + trow;
            const bf16x8 dta = cat8(lds_read_tr(dt + tile_off<D>(r0, db * 32 + tcol)),
                                    lds_read_tr(dt + tile_off<D>(r0 + 8, db * 32 + tcol)));
            const bf16x8 qta = cat8(lds_read_tr(qt + tile_off<D>(r0, db * 32 + tcol)),
                                    lds_read_tr(qt + tile_off<D>(r0 + 8, db * 32 + tcol)));
            dv[db] = mfma32(dta, pb[qb][c2], dv[db]);
            dk[db] = mfma32(qta, sb[qb][c2], dk[db]);
          }
    }
    cp.advance(BQ);
    if (t + 1 < T) store_step(buf ^ 1);
    __syncthreads();
    if (t + 2 < T) load_step();
  }

  if (!active) return;
  const int r = wkey0 + l32;
  if (r >= it.len) return;
  const int64_t ostride = int64_t(a.heads) * D;
  __bf16* krow = a.dk[s] + int64_t(it.start + r) * ostride + h * D;
  __bf16* vrow = a.dv[s] + int64_t(it.start + r) * ostride + h * D;
#pragma unroll
  for (int db = 0; db < ND; ++db)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 wk, wv;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        wk[e] = (__bf16)(dk[db][4 * g + e] * a.scale);
        wv[e] = (__bf16)(dv[db][4 * g + e]);
      }
      *reinterpret_cast<bf16x4*>(krow + db * 32 + 8 * g + 4 * half) = wk;
      *reinterpret_cast<bf16x4*>(vrow + db * 32 + 8 * g + 4 * half) = wv;
    }
}

hipError_t launch_dkv(const BwdArgs& a, int n_items, int head_dim, hipStream_t stream) {
  if (n_items <= 0) return hipSuccess;
  if (head_dim == 128)
    hipLaunchKernelGGL(sra_dkv_kernel<128>, dim3(n_items), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(sra_dkv_kernel<64>, dim3(n_items), dim3(kThreads), 0, stream, a);
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
