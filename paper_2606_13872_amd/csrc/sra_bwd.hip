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

// --------------------------------------------------------------------------- dkv
namespace {
constexpr int kDkvWaves = kDkvKeyTile / 32;
}

template <int D>
struct DkvState {
  bf16x8 vf[D / 16];    // V as B fragments (lane = key, 8 consecutive head dims)
  floatx16 dk[D / 32];  // dK^T accumulators (lane = key), 32 head dims each
  floatx16 dv[D / 32];  // dV^T accumulators
};

// One 32-query step for the wave's 32 keys. S = Q K^T and dP = dO V^T have lanes = keys and
// registers = query rows, so P and dS are directly the B fragments of dV^T += dO^T P and
// dK^T += Q^T dS. kMask: query rows >= nvalid are outside the span.
template <int D, bool kMask>
__device__ __forceinline__ void dkv_step(DkvState<D>& st, const __bf16* krow, const __bf16* qt,
                                         const __bf16* dt, const float* lse_s, const float* ndlt_s,
                                         int nvalid, float sl2) {
  constexpr int NC = D / 16, ND = D / 32, RQ = kRowPadRS<D>;  // Q and dO rows permuted
  const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
  const int qrow = perm16(l32);
  // dP starts from -D (staged negated in LDS, read in the accumulator's row order), so the
  // MFMAs leave dP - D and dS = P * (dP - D) is one multiply
  floatx16 s = floatx16{}, dp;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const floatx4 d4 = *reinterpret_cast<const floatx4*>(ndlt_s + 8 * g + 4 * half);
#pragma unroll
    for (int e = 0; e < 4; ++e) dp[4 * g + e] = d4[e];
  }
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const bf16x8 qa = *reinterpret_cast<const bf16x8*>(qt + qrow * RQ + c * 16 + half * 8);
    const bf16x8 kb = *reinterpret_cast<const bf16x8*>(krow + c * 16);
    const bf16x8 da = *reinterpret_cast<const bf16x8*>(dt + qrow * RQ + c * 16 + half * 8);
    s = mfma32(qa, kb, s);
    dp = mfma32(da, st.vf[c], dp);
  }
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int q0 = 8 * g + 4 * half;  // 4 consecutive query rows of this register group
    const floatx4 l4 = *reinterpret_cast<const floatx4*>(lse_s + q0);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int i = 4 * g + e;
      float p = fast_exp2(fmaf(s[i], sl2, -l4[e]));
      if constexpr (kMask) p = (q0 + e) < nvalid ? p : 0.f;
      s[i] = p;
      dp[i] = p * dp[i];
    }
  }
  // dV^T += dO^T P and dK^T += Q^T dS ; dO^T and Q^T fragments via the transpose read (rows
  // r0 and r0 + 8 sit at physical rows perm16(r0) and perm16(r0) + 2)
  const int tcol = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const int trow = 4 * half + ((lane & 15) >> 2);
#pragma unroll
  for (int c2 = 0; c2 < 2; ++c2) {
    const bf16x8 pb = to_bf16x8(s, 8 * c2);
    const bf16x8 sb = to_bf16x8(dp, 8 * c2);
    const int r0 = 16 * c2 + perm16(trow);
#pragma unroll
    for (int db = 0; db < ND; ++db) {
      const bf16x8 dta = cat8(lds_read_tr(dt + r0 * RQ + db * 32 + tcol),
                              lds_read_tr(dt + (r0 + 2) * RQ + db * 32 + tcol));
      st.dv[db] = mfma32(dta, pb, st.dv[db]);
      const bf16x8 qta = cat8(lds_read_tr(qt + r0 * RQ + db * 32 + tcol),
                              lds_read_tr(qt + (r0 + 2) * RQ + db * 32 + tcol));
      st.dk[db] = mfma32(qta, sb, st.dk[db]);
    }
  }
}

// Query tiles rotate through kDkvBufs LDS buffers and the workgroup meets at a barrier only
// after every second step, so the two waves of a SIMD can drift apart by up to a step and
// overlap one's softmax with the other's matrix products. Tiles are loaded two steps ahead.
// kOneStride: gen and ref q share one token stride, so one set of loader offsets serves both.
namespace {
constexpr int kDkvBufs = 4;
}

template <int D, bool kOneStride>
__global__ void __launch_bounds__(kDkvWaves * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
sra_dkv_kernel(BwdArgs a) {
  constexpr int NC = D / 16, ND = D / 32, BQ = kDkvQueryStep, RK = kRowPadRS<D>, RQ = kRowPadRS<D>;
  constexpr int NB = kDkvBufs;
  using KT = PaddedTile<D, kDkvKeyTile, RK>;
  using QT = PaddedTile<D, BQ, RQ>;
  __shared__ __attribute__((aligned(1024))) __bf16 ktile[KT::kElems];
  __shared__ __attribute__((aligned(1024))) __bf16 qs[NB][QT::kElems];
  __shared__ __attribute__((aligned(1024))) __bf16 dos[NB][QT::kElems];
  // per query row of a step: LSE (log2 units) in [0, BQ), -D in [BQ, 2 BQ)
  __shared__ __attribute__((aligned(16))) float rstat[NB][2 * BQ];

  const WorkItem it = a.items[blockIdx.x];
  if (it.stream < 0) return;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int half = lane >> 5, l32 = lane & 31;
  const int h = it.head, s = it.stream;
  const bool active = wave * 32 < it.len;
  const float sl2 = a.scale_log2;
  const int64_t dstride = int64_t(a.heads) * D;

  // the item's keys: K rows into LDS (clamped at the tile end), V fragments into VGPRs
  tile_load_lds<D, kDkvKeyTile, RK, kDkvWaves>(ktile, a.k[s], a.in_stride[s], h, it.start, it.len, 0, wave);
  DkvState<D> st;
  const int r = wave * 32 + l32;
  {
    const __bf16* vp = a.v[s] + int64_t(it.start + min(r, it.len - 1)) * a.in_stride[s] + h * D + half * 8;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const bf16x8 y = *reinterpret_cast<const bf16x8*>(vp + c * 16);
      st.vf[c] = (r < it.len) ? y : bf16x8{};
    }
#pragma unroll
    for (int db = 0; db < ND; ++db) {
      st.dk[db] = floatx16{};
      st.dv[db] = floatx16{};
    }
  }
  const __bf16* krow = ktile + r * RK + half * 8;

  const Span* sp = a.spans + it.span_off;
  const int T = count_steps(sp, it.span_cnt, BQ);
  SpanCursor ld;
  ld.init(sp, it.span_cnt);
  constexpr int NL = kOneStride ? 1 : 2;
  TileLoader<D, BQ, RQ, kDkvWaves, true> ql[NL], dl;  // Q and dO rows permuted
#pragma unroll
  for (int ss = 0; ss < NL; ++ss) ql[ss].init(a.in_stride[ss], h, wave);
  dl.init(dstride, h, wave);
  // wave 0 copies the step's row statistics straight into LDS: lanes < 32 the LSE, the
  // others -D (one row each, clamped at the span end like the tiles)
  static_assert(BQ == 32, "one dword per lane covers both statistics of 32 rows");
  auto issue = [&](int b) {  // the next step in the cursor -> buffer b
    const int ss = ld.stream();
    if (ld.off + BQ <= ld.len()) {
      const int64_t row0 = int64_t(ld.start() + ld.off);
      if (kOneStride || ss == 0)
        ql[0].issue(qs[b], a.q[ss] + row0 * a.in_stride[ss], wave);
      else
        ql[NL - 1].issue(qs[b], a.q[1] + row0 * a.in_stride[1], wave);
      dl.issue(dos[b], a.dout[ss] + row0 * dstride, wave);
    } else {
      tile_load_lds<D, BQ, RQ, kDkvWaves, true>(qs[b], a.q[ss], a.in_stride[ss], h, ld.start(), ld.len(), ld.off, wave);
      tile_load_lds<D, BQ, RQ, kDkvWaves, true>(dos[b], a.dout[ss], dstride, h, ld.start(), ld.len(), ld.off, wave);
    }
    if (wave == 0) {
      const int rr = ld.start() + min(ld.off + l32, ld.len() - 1);
      // both bases as uniform values first: a per-lane select of the argument slots would
      // become a vector load of the pointer and a wait on every load in flight
      const uint64_t pl = uniform_u64(reinterpret_cast<uint64_t>(a.lse2[ss]));
      const uint64_t pn = uniform_u64(reinterpret_cast<uint64_t>(a.ndelta[ss]));
      const float* src = reinterpret_cast<const float*>(half ? pn : pl);
      lds_dma_x1(src + int64_t(h) * a.rows[ss] + rr, rstat[b]);
    }
    ld.advance(BQ);
  };

  issue(0);
  if (T > 1) issue(1);
  wait_vmem();
  __syncthreads();
  // step t reads buffer t % NB and loads step t + 2 into buffer (t + 2) % NB, whose last
  // reader (step t - 2) finished before the barrier that ended step t - 1 or t - 2.
  auto step_tail = [&](int t) {
    if (t & 1) {  // every odd step: land the loads of steps t + 1 and t + 2, then meet
      wait_vmem();
      __syncthreads();
    }
  };
  int t = 0;
  for (int si = 0; si < it.span_cnt; ++si) {
    const int len = __builtin_amdgcn_readfirstlane(sp[si].len);
    const int full = len / BQ;
    for (int j = 0; j < full; ++j, ++t) {
      const int b = t % NB;
      if (t + 2 < T) issue((t + 2) % NB);
      if (active) dkv_step<D, false>(st, krow, qs[b], dos[b], rstat[b], rstat[b] + BQ, BQ, sl2);
      step_tail(t);
    }
    if (len % BQ) {
      const int b = t % NB;
      if (t + 2 < T) issue((t + 2) % NB);
      if (active) dkv_step<D, true>(st, krow, qs[b], dos[b], rstat[b], rstat[b] + BQ, len % BQ, sl2);
      step_tail(t);
      ++t;
    }
  }

  if (!active || r >= it.len) return;
  __bf16* kout = a.dk[s] + int64_t(it.start + r) * dstride + h * D;
  __bf16* vout = a.dv[s] + int64_t(it.start + r) * dstride + h * D;
#pragma unroll
  for (int db = 0; db < ND; ++db)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 wk, wv;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        wk[e] = (__bf16)(st.dk[db][4 * g + e] * a.scale);
        wv[e] = (__bf16)(st.dv[db][4 * g + e]);
      }
      *reinterpret_cast<bf16x4*>(kout + db * 32 + 8 * g + 4 * half) = wk;
      *reinterpret_cast<bf16x4*>(vout + db * 32 + 8 * g + 4 * half) = wv;
    }
}

hipError_t launch_dkv(const BwdArgs& a, int n_items, int head_dim, hipStream_t stream) {
  if (n_items <= 0) return hipSuccess;
  const bool one = a.in_stride[0] == a.in_stride[1];
  const dim3 grid(n_items), block(kDkvWaves * 64);
  if (head_dim == 128) {
    if (one) hipLaunchKernelGGL((sra_dkv_kernel<128, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((sra_dkv_kernel<128, false>), grid, block, 0, stream, a);
  } else {
    if (one) hipLaunchKernelGGL((sra_dkv_kernel<64, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((sra_dkv_kernel<64, false>), grid, block, 0, stream, a);
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
