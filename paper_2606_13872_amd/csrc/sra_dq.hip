// dQ kernel of the SRA backward on gfx950 (the gradient is described in sra_bwd.hip).
//
// Query-major, like the forward: a work item is a tile of 256 query rows of one stream and
// head; its four waves (one per SIMD) own 64 rows each, as two 32-row MFMA blocks, and keep
// those rows' Q and dO as B fragments in VGPRs and their dQ sums in AGPRs. The key rows the
// queries see (the spans of the query-major schedule) stream through LDS 32 at a time, and S
// and P are recomputed from the forward's log-sum-exp:
//     S^T = K Q^T, dP^T = V dO^T, dS^T = P^T (dP^T - D), dQ^T += K^T dS^T.
// Each K and V fragment read from LDS feeds both row blocks of a wave. Built with MFMAs in VGPR
// form; the dQ products are AGPR-accumulating MFMAs (mfma32_agpr).
#include "sra_kernels.h"
#include "sra_tiles.h"

namespace sra {

namespace {
constexpr int kDqWaves = kDqQueryTile / 64;  // one wave per SIMD, 64 query rows each
constexpr int kDqBufs = 4;
}

template <int D>
struct DqState {
  bf16x8 qf[2][D / 16];    // Q^T B fragments of the two row blocks (lane = query)
  bf16x8 df[2][D / 16];    // dO^T B fragments
  floatx16 dq[2][D / 32];  // dQ^T accumulators (lane = query), 32 head dims each
  float lse2[2], ndlt[2];  // the rows' log-sum-exp (log2 units) and -rowsum(dO * O)
};

// One 32-key step for the wave's 64 query rows. S^T and dP^T have lanes = queries and
// registers = keys, so dS^T is directly the B fragment of dQ^T += K^T dS^T. Three phases of NC
// slots (S, dP, dQ); each slot issues the LDS reads of the next slot, its MFMAs and a share of
// the VALU work (dP's starting value -D during S, the exponentials during dP, the second half
// of dS during dQ), and ends at a scheduling barrier. kMask: keys >= nvalid are outside the span.
template <int D, bool kMask>
__device__ __forceinline__ void dq_step(DqState<D>& st, const __bf16* kt, const __bf16* vt, int nvalid,
                                        float sl2) {
  constexpr int NC = D / 16, ND = D / 32, RK = kBothPadRS<D>, RV = kRowPadRS<D>;
  constexpr int EP = 32 / NC;  // P elements per dP slot over both blocks
  constexpr int IP = 16 / NC;  // dP registers set to -D per S slot and block
  const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
  const __bf16* ka_p = kt + l32 * RK + half * 8;
  const __bf16* va_p = vt + l32 * RV + half * 8;
  // K^T fragments through the transpose read: key rows r0 and r0 + 8 of each 16-key half
  const int toff = (4 * half + ((lane & 15) >> 2)) * RK + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
#define SRA_TR(j) \
  cat8(lds_read_tr(kt + toff + (16 * ((j) / ND)) * RK + ((j) % ND) * 32), \
       lds_read_tr(kt + toff + (16 * ((j) / ND) + 8) * RK + ((j) % ND) * 32))

  // ---- S^T, while dP^T is set to -D
  floatx16 s0 = floatx16{}, s1 = floatx16{}, dp0, dp1;
  bf16x8 ka = ld8(ka_p), va;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    bf16x8 nk;
    if (c + 1 < NC) nk = ld8(ka_p + (c + 1) * 16);
    else va = ld8(va_p);
    s0 = mfma32(ka, st.qf[0][c], s0);
    s1 = mfma32(ka, st.qf[1][c], s1);
#pragma unroll
    for (int u = 0; u < IP; ++u) {
      dp0[c * IP + u] = st.ndlt[0];
      dp1[c * IP + u] = st.ndlt[1];
    }
    __builtin_amdgcn_sched_barrier(0);
    if (c + 1 < NC) ka = nk;
  }
  // ---- dP^T, with P^T = exp2(S^T scale log2e - LSE) of both blocks
  bf16x8 tf;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    bf16x8 nv;
    if (c + 1 < NC) nv = ld8(va_p + (c + 1) * 16);
    else tf = SRA_TR(0);
    dp0 = mfma32(va, st.df[0][c], dp0);
    dp1 = mfma32(va, st.df[1][c], dp1);
#pragma unroll
    for (int u = 0; u < EP; ++u) {
      const int x = c * EP + u, i = x % 16, key = 8 * (i / 4) + 4 * half + (i % 4);
      if (x < 16) {
        float p = fast_exp2(fmaf(s0[i], sl2, -st.lse2[0]));
        if constexpr (kMask) p = key < nvalid ? p : 0.f;
        s0[i] = p;
      } else {
        float p = fast_exp2(fmaf(s1[i], sl2, -st.lse2[1]));
        if constexpr (kMask) p = key < nvalid ? p : 0.f;
        s1[i] = p;
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    if (c + 1 < NC) va = nv;
  }
  // ---- dQ^T += K^T dS^T; dS of the first 16 keys before, of the last 16 during the products
  bf16x8 dsf[2][2];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    dp0[i] = s0[i] * dp0[i];
    dp1[i] = s1[i] * dp1[i];
  }
  dsf[0][0] = to_bf16x8(dp0, 0);
  dsf[1][0] = to_bf16x8(dp1, 0);
  constexpr int EQ = 8 / ND;  // second-half dS elements per block per slot of the first half
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    const int c2 = j / ND, db = j % ND;
    bf16x8 nx;
    if (j + 1 < NC) nx = SRA_TR(j + 1);
    mfma32_agpr(st.dq[0][db], tf, dsf[0][c2]);
    mfma32_agpr(st.dq[1][db], tf, dsf[1][c2]);
    if (j < ND) {
#pragma unroll
      for (int u = 0; u < EQ; ++u) {
        const int i = 8 + j * EQ + u;
        dp0[i] = s0[i] * dp0[i];
        dp1[i] = s1[i] * dp1[i];
      }
      if (j == ND - 1) {
        dsf[0][1] = to_bf16x8(dp0, 8);
        dsf[1][1] = to_bf16x8(dp1, 8);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    if (j + 1 < NC) tf = nx;
  }
#undef SRA_TR
}

template <int D>
__global__ void __launch_bounds__(kDqWaves * 64) __attribute__((amdgpu_waves_per_eu(1, 1)))
sra_dq_kernel(BwdArgs a) {
  constexpr int NC = D / 16, ND = D / 32, BK = kDqKeyStep, RK = kBothPadRS<D>, RV = kRowPadRS<D>;
  // K is read both as row fragments and through the transpose read, from one copy at D + 24.
  // Key tiles rotate through kDqBufs buffers, are loaded two steps ahead, and the workgroup
  // meets at a barrier after every second step.
  constexpr int NB = kDqBufs;
  using KT = PaddedTile<D, BK, RK>;
  using VT = PaddedTile<D, BK, RV>;
  __shared__ __attribute__((aligned(1024))) __bf16 ks[NB][KT::kElems];
  __shared__ __attribute__((aligned(1024))) __bf16 vs[NB][VT::kElems];

  const WorkItem it = a.items[blockIdx.x];
  if (it.stream < 0) return;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int half = lane >> 5, l32 = lane & 31;
  const int h = it.head, s = it.stream;
  const bool active = wave * 64 < it.len;
  const float sl2 = a.scale_log2;
  const int64_t dstride = int64_t(a.heads) * D;

  DqState<D> st;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int r = wave * 64 + 32 * j + l32;
    const int rr = it.start + min(r, it.len - 1);
    const __bf16* qp = a.q[s] + int64_t(rr) * a.in_stride[s] + h * D + half * 8;
    const __bf16* dp = a.dout[s] + int64_t(rr) * dstride + h * D + half * 8;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const bf16x8 x = ld8(qp + c * 16);
      const bf16x8 y = ld8(dp + c * 16);
      st.qf[j][c] = (r < it.len) ? x : bf16x8{};
      st.df[j][c] = (r < it.len) ? y : bf16x8{};
    }
#pragma unroll
    for (int db = 0; db < ND; ++db) st.dq[j][db] = floatx16{};
    st.lse2[j] = a.lse2[s][int64_t(h) * a.rows[s] + rr];
    st.ndlt[j] = a.ndelta[s][int64_t(h) * a.rows[s] + rr];
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
  // per-stream bases and LDS byte addresses as uniform scalars
  const uint64_t kb0 = uniform_u64(reinterpret_cast<uint64_t>(a.k[0]));
  const uint64_t kb1 = uniform_u64(reinterpret_cast<uint64_t>(a.k[1]));
  const uint64_t vb0 = uniform_u64(reinterpret_cast<uint64_t>(a.v[0]));
  const uint64_t vb1 = uniform_u64(reinterpret_cast<uint64_t>(a.v[1]));
  const int64_t st0 = a.in_stride[0], st1 = a.in_stride[1];
  constexpr uint32_t kKBytes = KT::kElems * 2, kVBytes = VT::kElems * 2;
  constexpr int kKFull = KT::kInstr / kDqWaves, kVFull = VT::kInstr / kDqWaves;
  const bool k_extra = wave + kKFull * kDqWaves < KT::kInstr;
  const bool v_extra = wave + kVFull * kDqWaves < VT::kInstr;
  const uint32_t k_lds = lds_addr(&ks[0][0]) + wave * 1024, v_lds = lds_addr(&vs[0][0]) + wave * 1024;
  auto issue = [&](int b) __attribute__((always_inline)) {  // the next step -> buffer b
    const int ss = ld.stream();
    if (ld.off + BK <= ld.len()) {
      const int64_t row0 = int64_t(ld.start() + ld.off) * (ss ? st1 : st0);
      const __bf16* kg = reinterpret_cast<const __bf16*>(ss ? kb1 : kb0) + row0;
      const __bf16* vg = reinterpret_cast<const __bf16*>(ss ? vb1 : vb0) + row0;
      const uint32_t ka = k_lds + b * kKBytes, va = v_lds + b * kVBytes;
#pragma unroll
      for (int j = 0; j < kKFull + 1; ++j)
        if (j < kKFull || k_extra) lds_dma_x4_at(kg + (ss ? kl[1].voff[j] : kl[0].voff[j]), ka + j * kDqWaves * 1024);
#pragma unroll
      for (int j = 0; j < kVFull + 1; ++j)
        if (j < kVFull || v_extra) lds_dma_x4_at(vg + (ss ? vl[1].voff[j] : vl[0].voff[j]), va + j * kDqWaves * 1024);
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
  auto step_tail = [&](int t) {
    if (t & 1) {
      wait_vmem();
      __syncthreads();
    }
    if (t + 1 == T) mfma_drain();
  };
  int t = 0;
  for (int si = 0; si < it.span_cnt; ++si) {
    const int len = __builtin_amdgcn_readfirstlane(sp[si].len);
    const int full = len / BK;
    for (int j = 0; j < full; ++j, ++t) {
      if (t + 2 < T) issue((t + 2) % NB);
      if (active) dq_step<D, false>(st, ks[t % NB], vs[t % NB], BK, sl2);
      step_tail(t);
    }
    if (len % BK) {
      if (t + 2 < T) issue((t + 2) % NB);
      if (active) dq_step<D, true>(st, ks[t % NB], vs[t % NB], len % BK, sl2);
      step_tail(t);
      ++t;
    }
  }

  if (!active) return;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int r = wave * 64 + 32 * j + l32;
    if (r >= it.len) continue;
    __bf16* orow = a.dq[s] + int64_t(it.start + r) * dstride + h * D;
#pragma unroll
    for (int db = 0; db < ND; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = (__bf16)(st.dq[j][db][4 * g + e] * a.scale);
        *reinterpret_cast<bf16x4*>(orow + db * 32 + 8 * g + 4 * half) = w;
      }
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
