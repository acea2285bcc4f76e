// Forward pass of Sparse Reference Attention on gfx950.
//
// One workgroup (8 wave64s, two per SIMD) takes one work item: a tile of up to 256 query
// rows of one stream and head, plus the list of key spans those rows see (Avatar V §1,
// §2.1, §4.3: gen rows see the gen keys and the valid ref frames of their sample; ref rows
// see the valid frames of their own group). Keys stream through LDS 64 rows at a time with
// direct global->LDS loads into two buffers; every wave owns 32 query rows, and the two
// waves of a SIMD overlap one's softmax (VALU) with the other's matrix products:
//
//   S^T (keys x queries) = K Q^T          bf16 MFMA 32x32x16, K rows from LDS, Q^T in VGPRs
//   online softmax over keys in base 2, lanes = queries (row sums are lane-local plus one
//   permlane32 swap); the running max is only recomputed when P would exceed 2^16, which
//   the partial row sums detect, so the common step does no max at all and rescaling is rare
//   O^T (d x queries) += V^T P^T          V^T fragments via the LDS transpose read
//
// Only the last step of a span (its ragged tail) runs the masked variant of the step;
// there is no dense mask.
#include "sra_kernels.h"
#include "sra_tiles.h"

namespace sra {

namespace {
constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kBigSum = 65536.0f;    // a lane's step sum of P above this forces a rescale
constexpr int kWaves = kFwdQueryTile / 32;
template <int D> using KTile = PaddedTile<D, kFwdKeyStep, kRowPadRS<D>>;  // row-fragment reads
template <int D> using VTile = PaddedTile<D, kFwdKeyStep, kTrPadRS<D>>;   // transpose reads
}  // namespace

template <int D>
struct FwdState {
  bf16x8 qf[D / 16];   // Q^T MFMA B fragments: lane = query, 8 consecutive head dims
  floatx16 o[D / 32];  // O^T accumulators, 32 head dims each
  float m;             // running max (log2 units)
  float l;             // per-lane partial row sum (fp32)
};

// S^T (keys x queries) of the 64 keys at kt for the wave's 32 query rows; keys >= nvalid are
// outside the span (kMask).
template <int D, bool kMask>
__device__ __forceinline__ void fwd_scores(const FwdState<D>& st, const __bf16* kt, int nvalid, floatx16& s0,
                                           floatx16& s1) {
  constexpr int NC = D / 16;
  const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
  s0 = floatx16{};
  s1 = floatx16{};
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(kt + l32 * kRowPadRS<D> + c * 16 + half * 8);
    const bf16x8 k1 = *reinterpret_cast<const bf16x8*>(kt + (32 + l32) * kRowPadRS<D> + c * 16 + half * 8);
    s0 = mfma32(k0, st.qf[c], s0);
    s1 = mfma32(k1, st.qf[c], s1);
  }
  if constexpr (kMask) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int key = 8 * (i >> 2) + 4 * half + (i & 3);
      s0[i] = key >= nvalid ? -INFINITY : s0[i];
      s1[i] = key + 32 >= nvalid ? -INFINITY : s1[i];
    }
  }
}

// P = exp2(S * scale*log2e - m) in place; returns this lane's partial row sum.
__device__ __forceinline__ float fwd_exp(floatx16& s0, floatx16& s1, float m, float sl2) {
  const float nm = -m;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};  // 4 independent partial sums
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    s0[i] = fast_exp2(fmaf(s0[i], sl2, nm));
    s1[i] = fast_exp2(fmaf(s1[i], sl2, nm));
    acc[i & 3] += s0[i] + s1[i];
  }
  return (acc[0] + acc[1]) + (acc[2] + acc[3]);
}

// One 64-key step for the wave's 32 query rows. kMask: keys >= nvalid are outside the span.
//
// The running max m is not tracked per step. P is computed against the current m, and its
// partial row sum doubles as the overflow check: if some lane's 32 values sum to more than
// kBigSum (some P > kBigSum, or an inf from m = -inf on the first step), the wave takes the
// rare slow path: recompute S, set m to the true running max, rescale O and l, recompute P.
// So m always lies within log2(kBigSum) of the true row max, which bounds every P by kBigSum.
template <int D, bool kMask>
__device__ __forceinline__ void fwd_step(FwdState<D>& st, const __bf16* kt, const __bf16* vt, int nvalid,
                                         float sl2) {
  constexpr int ND = D / 32;
  const int lane = threadIdx.x & 63, half = lane >> 5;
  floatx16 s0, s1;  // S^T for keys 0..31 and 32..63, then P
  fwd_scores<D, kMask>(st, kt, nvalid, s0, s1);
  float lsum = fwd_exp(s0, s1, st.m, sl2);
  if (__builtin_expect(__builtin_amdgcn_ballot_w64(!(lsum <= kBigSum)) != 0, 0)) {
    fwd_scores<D, kMask>(st, kt, nvalid, s0, s1);
    float mq[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) mq[j] = max3f(max2f(s0[4 * j], s1[4 * j]), s0[4 * j + 1], s1[4 * j + 1]);
#pragma unroll
    for (int j = 0; j < 4; ++j) mq[j] = max3f(mq[j], max3f(s0[4 * j + 2], s1[4 * j + 2], s0[4 * j + 3]), s1[4 * j + 3]);
    const float mx = pair_max(max2f(max2f(mq[0], mq[1]), max2f(mq[2], mq[3]))) * sl2;
    if (mx > st.m) {
      const float alpha = fast_exp2(st.m - mx);  // 0 when m was -inf
      st.m = mx;
      st.l *= alpha;
#pragma unroll
      for (int db = 0; db < ND; ++db) st.o[db] *= alpha;
    }
    lsum = fwd_exp(s0, s1, st.m, sl2);
  }
  st.l += lsum;
  // O^T += V^T P^T: the transpose read gives lane (head dim l32) the 8 keys whose P values
  // the B fragment holds, in the MFMA output's register order.
  const int tcol = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const int trow = 4 * half + ((lane & 15) >> 2);
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2) {
      const bf16x8 p = to_bf16x8(kb ? s1 : s0, 8 * c2);
      const int r0 = kb * 32 + 16 * c2 + trow;
#pragma unroll
      for (int db = 0; db < ND; ++db) {
        const bf16x8 va = cat8(lds_read_tr(vt + r0 * kTrPadRS<D> + db * 32 + tcol),
                               lds_read_tr(vt + (r0 + 8) * kTrPadRS<D> + db * 32 + tcol));
        st.o[db] = mfma32(va, p, st.o[db]);
      }
    }
}

template <int D>
__global__ void __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
sra_fwd_kernel(FwdArgs a) {
  constexpr int NC = D / 16, ND = D / 32, BK = kFwdKeyStep;
  __shared__ __attribute__((aligned(1024))) __bf16 ks[2][KTile<D>::kElems];
  __shared__ __attribute__((aligned(1024))) __bf16 vs[2][VTile<D>::kElems];

  const WorkItem it = a.items[blockIdx.x];
  if (it.stream < 0) return;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int half = lane >> 5, l32 = lane & 31;
  const int h = it.head, s = it.stream;
  const int wrow0 = wave * 32;
  const bool active = wrow0 < it.len;
  const float sl2 = a.scale_log2;

  FwdState<D> st;
  const int r = wrow0 + l32;
  {
    const __bf16* src = a.q[s] + int64_t(it.start + min(r, it.len - 1)) * a.in_stride[s] + h * D + half * 8;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const bf16x8 x = *reinterpret_cast<const bf16x8*>(src + c * 16);
      st.qf[c] = (r < it.len) ? x : bf16x8{};
    }
#pragma unroll
    for (int db = 0; db < ND; ++db) st.o[db] = floatx16{};
    st.m = -INFINITY;
    st.l = 0.f;
  }

  const Span* sp = a.spans + it.span_off;
  const int T = count_steps(sp, it.span_cnt, BK);
  SpanCursor ld;
  ld.init(sp, it.span_cnt);
  TileLoader<D, BK, kRowPadRS<D>, kWaves> kl[2];
  TileLoader<D, BK, kTrPadRS<D>, kWaves> vl[2];
#pragma unroll
  for (int ss = 0; ss < 2; ++ss) {
    kl[ss].init(a.in_stride[ss], h, wave);
    vl[ss].init(a.in_stride[ss], h, wave);
  }
  auto issue = [&](int b) {
    const int ss = ld.stream();
    if (ld.off + BK <= ld.len()) {  // whole tile inside the span: fixed lane offsets
      const int64_t row0 = int64_t(ld.start() + ld.off) * a.in_stride[ss];
      if (ss == 0) {
        kl[0].issue(ks[b], a.k[0] + row0, wave);
        vl[0].issue(vs[b], a.v[0] + row0, wave);
      } else {
        kl[1].issue(ks[b], a.k[1] + row0, wave);
        vl[1].issue(vs[b], a.v[1] + row0, wave);
      }
    } else {
      tile_load_lds<D, BK, kRowPadRS<D>, kWaves>(ks[b], a.k[ss], a.in_stride[ss], h, ld.start(), ld.len(), ld.off, wave);
      tile_load_lds<D, BK, kTrPadRS<D>, kWaves>(vs[b], a.v[ss], a.in_stride[ss], h, ld.start(), ld.len(), ld.off, wave);
    }
    ld.advance(BK);
  };

  issue(0);
  wait_vmem();
  __syncthreads();
  // Steps are numbered t over the whole span list (two LDS buffers alternate). Full steps of
  // a span and its ragged last step run in separate loops, so the unmasked step carries no
  // masking code at all.
  int t = 0;
  for (int si = 0; si < it.span_cnt; ++si) {
    const int len = __builtin_amdgcn_readfirstlane(sp[si].len);
    const int full = len / BK;
    for (int j = 0; j < full; ++j, ++t) {
      if (t + 1 < T) issue((t + 1) & 1);
      if (active) fwd_step<D, false>(st, ks[t & 1], vs[t & 1], BK, sl2);
      wait_vmem();
      __syncthreads();
    }
    if (len % BK) {
      if (t + 1 < T) issue((t + 1) & 1);
      if (active) fwd_step<D, true>(st, ks[t & 1], vs[t & 1], len % BK, sl2);
      wait_vmem();
      __syncthreads();
      ++t;
    }
  }

  if (!active) return;
  const int64_t ostride = int64_t(a.heads) * D;
  const float lt = pair_sum(st.l);
  const float inv = 1.f / lt;
  if (r < it.len) {
    __bf16* orow = a.o[s] + int64_t(it.start + r) * ostride + h * D;
#pragma unroll
    for (int db = 0; db < ND; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = (__bf16)(st.o[db][4 * g + e] * inv);
        *reinterpret_cast<bf16x4*>(orow + db * 32 + 8 * g + 4 * half) = w;
      }
    if (half == 0) a.lse[s][int64_t(h) * a.rows[s] + it.start + r] = (st.m + log2f(lt)) * kLn2;
  }
}

hipError_t launch_forward(const FwdArgs& a, int n_items, int head_dim, hipStream_t stream) {
  if (n_items <= 0) return hipSuccess;
  if (head_dim == 128)
    hipLaunchKernelGGL(sra_fwd_kernel<128>, dim3(n_items), dim3(kWaves * 64), 0, stream, a);
  else
    hipLaunchKernelGGL(sra_fwd_kernel<64>, dim3(n_items), dim3(kWaves * 64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace sra
