// dQ kernel of the SRA backward on gfx950 (the gradient is described in sra_bwd.hip).
//
// Query-major, like the forward: a work item is a tile of 256 query rows of one stream and
// head; it streams the key rows those queries see (the spans of the query-major schedule)
// through LDS 32 at a time and recomputes S and P from the forward's log-sum-exp:
//     S^T = K Q^T, dP^T = V dO^T, dS^T = P^T (dP^T - D), dQ^T += K^T dS^T.
#include "sra_kernels.h"
#include "sra_tiles.h"

namespace sra {

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


}  // namespace sra
