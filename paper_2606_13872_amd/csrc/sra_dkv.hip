// dK/dV kernel of the SRA backward on gfx950 (the gradient is described in sra_bwd.hip).
//
// Key-major: a work item is a tile of 256 keys of one stream and head; its four waves (one per
// SIMD) own 64 keys each, as two 32-key MFMA blocks, and keep those keys' V in VGPRs and their
// dK and dV sums in AGPRs for the whole item. K sits in LDS. The query rows that see the keys
// stream through LDS 32 at a time (gen keys: the gen queries of the sample; ref keys: the gen
// queries plus the ref queries of the key's group; a tile may hold keys of two groups, and
// then each group's query span reaches only its own range of the tile's keys):
//     S = Q K^T, dP = dO V^T, P = exp2(S scale log2e - LSE), dS = P (dP - D),
//     dV^T += dO^T P, dK^T += Q^T dS.
// Each Q and dO fragment read from LDS feeds both key blocks of a wave, which halves the LDS
// reads per product against one 32-key block per wave. Built with MFMAs in VGPR form (S and dP
// live in VGPRs); the dK/dV products are written as AGPR-accumulating MFMAs (mfma32_agpr).
#include "sra_kernels.h"
#include "sra_tiles.h"

namespace sra {

namespace {
constexpr int kDkvWaves = kDkvKeyTile / 64;  // one wave per SIMD, 64 keys (two 32-key blocks) each
constexpr int kDkvBufs = 4;
}

template <int D>
struct DkvState {
  bf16x8 vf[2][D / 16];    // V of the wave's two key blocks as B fragments (lane = key)
  floatx16 dk[2][D / 32];  // dK^T accumulators (lane = key), 32 head dims each
  floatx16 dv[2][D / 32];  // dV^T accumulators
};

// One 32-query step for the wave's 64 keys. S = Q K^T and dP = dO V^T have lanes = keys and
// registers = query rows, so P and dS are directly the B fragments of dV^T += dO^T P and
// dK^T += Q^T dS; each Q and dO fragment read from LDS feeds both key blocks. The products
// run in four phases of NC slots (S, dP, dV, dK); each slot issues the LDS reads of the next
// slot, two MFMAs and a share of the VALU work (the exponentials during dP, dS during dV),
// and ends at a scheduling barrier so the compiler keeps that interleave and the register
// footprint of one slot. kMask: query rows >= nvalid are outside the span, and the lane's key of
// block j takes part only if kvj (a span that reaches only part of the tile's keys).
template <int D, bool kMask>
__device__ __forceinline__ void dkv_step(DkvState<D>& st, const __bf16* krow, const __bf16* qt,
                                         const __bf16* dt, const float* lse_s, const float* ndlt_s,
                                         int nvalid, float sl2, bool kv0 = true, bool kv1 = true) {
  constexpr int NC = D / 16, ND = D / 32, RQ = kRowPadRS<D>, RK = kRowPadRS<D>;  // Q, dO rows permuted
  constexpr int EP = 32 / NC;  // P (or dS) elements per slot, over both blocks
  const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
  const __bf16* qa_p = qt + perm16(l32) * RQ + half * 8;
  const __bf16* da_p = dt + perm16(l32) * RQ + half * 8;
  // transpose reads: rows r0 and r0 + 8 of a 16-row block sit at physical rows perm16(r0) and
  // perm16(r0) + 2
  const int tcol = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const int toff = perm16(4 * half + ((lane & 15) >> 2)) * RQ + tcol;
#define SRA_TR(base, j) \
  cat8(lds_read_tr((base) + toff + (16 * ((j) / ND)) * RQ + ((j) % ND) * 32), \
       lds_read_tr((base) + toff + (16 * ((j) / ND) + 2) * RQ + ((j) % ND) * 32))

  // ---- S
  floatx16 s0 = floatx16{}, s1 = floatx16{}, dp0, dp1;
  floatx4 l4[4];
  bf16x8 qa = ld8(qa_p), k0 = ld8(krow), k1 = ld8(krow + 32 * RK), da;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    bf16x8 nq, nk0, nk1;
    if (c + 1 < NC) {
      nq = ld8(qa_p + (c + 1) * 16);
      nk0 = ld8(krow + (c + 1) * 16);
      nk1 = ld8(krow + 32 * RK + (c + 1) * 16);
    } else {
      da = ld8(da_p);
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        l4[g] = *reinterpret_cast<const floatx4*>(lse_s + 8 * g + 4 * half);
        // dP starts from -D, so the products leave dP - D
        const floatx4 d4 = *reinterpret_cast<const floatx4*>(ndlt_s + 8 * g + 4 * half);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          dp0[4 * g + e] = d4[e];
          dp1[4 * g + e] = d4[e];
        }
      }
    }
    s0 = mfma32(qa, k0, s0);
    s1 = mfma32(qa, k1, s1);
    __builtin_amdgcn_sched_barrier(0);
    if (c + 1 < NC) {
      qa = nq;
      k0 = nk0;
      k1 = nk1;
    }
  }
  // ---- dP, with P = exp2(S scale log2e - LSE) of both blocks
  bf16x8 pb[2][2], sb[2][2], tf;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    bf16x8 nd;
    if (c + 1 < NC) nd = ld8(da_p + (c + 1) * 16);
    else tf = SRA_TR(dt, 0);
    dp0 = mfma32(da, st.vf[0][c], dp0);
    dp1 = mfma32(da, st.vf[1][c], dp1);
#pragma unroll
    for (int u = 0; u < EP; ++u) {
      const int x = c * EP + u, i = x % 16, q = 8 * (i / 4) + 4 * half + (i % 4);
      if (x < 16) {
        float p = fast_exp2(fmaf(s0[i], sl2, -l4[i / 4][i % 4]));
        if constexpr (kMask) p = (q < nvalid && kv0) ? p : 0.f;
        s0[i] = p;
      } else {
        float p = fast_exp2(fmaf(s1[i], sl2, -l4[i / 4][i % 4]));
        if constexpr (kMask) p = (q < nvalid && kv1) ? p : 0.f;
        s1[i] = p;
      }
    }
#pragma unroll
    for (int gi = 0; gi < 4; ++gi)  // 8-element groups completed in this slot
      if (8 * gi + 8 <= (c + 1) * EP && 8 * gi + 8 > c * EP)
        pb[gi / 2][gi % 2] = to_bf16x8(gi < 2 ? s0 : s1, 8 * (gi % 2));
    __builtin_amdgcn_sched_barrier(0);
    if (c + 1 < NC) da = nd;
  }
  // ---- dV^T += dO^T P, with dS = P (dP - D)
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    const int c2 = j / ND, db = j % ND;
    const bf16x8 nx = (j + 1 < NC) ? SRA_TR(dt, j + 1) : SRA_TR(qt, 0);
    mfma32_agpr(st.dv[0][db], tf, pb[0][c2]);
    mfma32_agpr(st.dv[1][db], tf, pb[1][c2]);
#pragma unroll
    for (int u = 0; u < EP; ++u) {
      const int x = j * EP + u, i = x % 16;
      if (x < 16) dp0[i] = s0[i] * dp0[i];
      else dp1[i] = s1[i] * dp1[i];
    }
#pragma unroll
    for (int gi = 0; gi < 4; ++gi)
      if (8 * gi + 8 <= (j + 1) * EP && 8 * gi + 8 > j * EP)
        sb[gi / 2][gi % 2] = to_bf16x8(gi < 2 ? dp0 : dp1, 8 * (gi % 2));
    __builtin_amdgcn_sched_barrier(0);
    tf = nx;
  }
  // ---- dK^T += Q^T dS
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    const int c2 = j / ND, db = j % ND;
    bf16x8 nx;
    if (j + 1 < NC) nx = SRA_TR(qt, j + 1);
    mfma32_agpr(st.dk[0][db], tf, sb[0][c2]);
    mfma32_agpr(st.dk[1][db], tf, sb[1][c2]);
    __builtin_amdgcn_sched_barrier(0);
    if (j + 1 < NC) tf = nx;
  }
#undef SRA_TR
}

// Query tiles rotate through kDkvBufs LDS buffers and the workgroup meets at a barrier only
// after every second step; tiles are loaded two steps ahead.
// kOneStride: gen and ref q share one token stride, so one set of loader offsets serves both.
template <int D, bool kOneStride>
__global__ void __launch_bounds__(kDkvWaves * 64) __attribute__((amdgpu_waves_per_eu(1, 1)))
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
  const bool active = wave * 64 < it.len;
  const float sl2 = a.scale_log2;
  const int64_t dstride = int64_t(a.heads) * D;

  // the item's keys: K rows into LDS (clamped at the tile end), V fragments into VGPRs
  tile_load_lds<D, kDkvKeyTile, RK, kDkvWaves>(ktile, a.k[s], a.in_stride[s], h, it.start, it.len, 0, wave);
  DkvState<D> st;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int r = wave * 64 + 32 * j + l32;
    const __bf16* vp = a.v[s] + int64_t(it.start + min(r, it.len - 1)) * a.in_stride[s] + h * D + half * 8;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const bf16x8 y = *reinterpret_cast<const bf16x8*>(vp + c * 16);
      st.vf[j][c] = (r < it.len) ? y : bf16x8{};
    }
#pragma unroll
    for (int db = 0; db < ND; ++db) {
      st.dk[j][db] = floatx16{};
      st.dv[j][db] = floatx16{};
    }
  }
  const __bf16* krow = ktile + (wave * 64 + l32) * RK + half * 8;

  const Span* sp = a.spans + it.span_off;
  const int T = count_steps(sp, it.span_cnt, BQ);
  SpanCursor ld;
  ld.init(sp, it.span_cnt);
  constexpr int NL = kOneStride ? 1 : 2;
  TileLoader<D, BQ, RQ, kDkvWaves, true> ql[NL], dl;  // Q and dO rows permuted (lane offsets)
#pragma unroll
  for (int ss = 0; ss < NL; ++ss) ql[ss].init(a.in_stride[ss], h, wave);
  dl.init(dstride, h, wave);
  // per-stream bases and LDS byte addresses as uniform scalars, so the loads of a step need
  // no argument reads
  const uint64_t qb0 = uniform_u64(reinterpret_cast<uint64_t>(a.q[0]));
  const uint64_t qb1 = uniform_u64(reinterpret_cast<uint64_t>(a.q[1]));
  const uint64_t db0 = uniform_u64(reinterpret_cast<uint64_t>(a.dout[0]));
  const uint64_t db1 = uniform_u64(reinterpret_cast<uint64_t>(a.dout[1]));
  const uint64_t lb0 = uniform_u64(reinterpret_cast<uint64_t>(a.lse2[0]));
  const uint64_t lb1 = uniform_u64(reinterpret_cast<uint64_t>(a.lse2[1]));
  const uint64_t nb0 = uniform_u64(reinterpret_cast<uint64_t>(a.ndelta[0]));
  const uint64_t nb1 = uniform_u64(reinterpret_cast<uint64_t>(a.ndelta[1]));
  const int64_t qst0 = a.in_stride[0], qst1 = a.in_stride[1];
  const int hr0 = h * a.rows[0], hr1 = h * a.rows[1];
  using QTL = PaddedTile<D, BQ, RQ>;
  constexpr uint32_t kBufBytes = QTL::kElems * 2;
  constexpr int kFull = QTL::kInstr / kDkvWaves;  // load slots every wave has
  const uint32_t q_lds = lds_addr(&qs[0][0]) + wave * 1024, d_lds = lds_addr(&dos[0][0]) + wave * 1024;
  const bool extra_slot = wave + kFull * kDkvWaves < QTL::kInstr;
  static_assert(BQ == 32, "one dword per lane covers both statistics of 32 rows");
  float stat = 0.f;  // the row statistics a wave loads for a later step (waves take turns)
  auto issue = [&](int b, int u) __attribute__((always_inline)) {  // step u -> buffer b
    const int ss = ld.stream();
    if (wave == (u & 3)) {  // lanes < 32: LSE of the step's rows; the others: -D
      const int rr = ld.start() + min(ld.off + l32, ld.len() - 1) + (ss ? hr1 : hr0);
      const uint64_t nbs = ss ? nb1 : nb0, lbs = ss ? lb1 : lb0;
      const uint64_t base = half ? nbs : lbs;
      stat = reinterpret_cast<const __attribute__((address_space(1))) float*>(base)[rr];
    }
    if (ld.off + BQ <= ld.len()) {
      const int64_t row0 = int64_t(ld.start() + ld.off);
      const __bf16* qg = reinterpret_cast<const __bf16*>(ss ? qb1 : qb0) + row0 * (ss ? qst1 : qst0);
      const __bf16* dg = reinterpret_cast<const __bf16*>(ss ? db1 : db0) + row0 * dstride;
      const uint32_t qa = q_lds + b * kBufBytes, da = d_lds + b * kBufBytes;
#pragma unroll
      for (int j = 0; j < kFull + 1; ++j) {
        if (j < kFull || extra_slot) {
          const int qo = (kOneStride || ss == 0) ? ql[0].voff[j] : ql[NL - 1].voff[j];
          lds_dma_x4_at(qg + qo, qa + j * kDkvWaves * 1024);
          lds_dma_x4_at(dg + dl.voff[j], da + j * kDkvWaves * 1024);
        }
      }
    } else {
      tile_load_lds<D, BQ, RQ, kDkvWaves, true>(qs[b], a.q[ss], a.in_stride[ss], h, ld.start(), ld.len(), ld.off, wave);
      tile_load_lds<D, BQ, RQ, kDkvWaves, true>(dos[b], a.dout[ss], dstride, h, ld.start(), ld.len(), ld.off, wave);
    }
    ld.advance(BQ);
  };
  // the loading wave stores the statistics of step u at the end of step u - 2 (they are read
  // at step u, after the barrier of step u - 2 or u - 1)
  auto put_stat = [&](int u) __attribute__((always_inline)) {
    if (wave == (u & 3)) rstat[u % NB][lane] = stat;
  };

  issue(0, 0);
  put_stat(0);
  if (T > 1) {
    issue(1, 1);
    put_stat(1);
  }
  wait_vmem();
  __syncthreads();
  // step t reads buffer t % NB and loads step t + 2 into buffer (t + 2) % NB, whose last
  // reader (step t - 2) finished before the barrier that ended step t - 1 or t - 2.
  auto step_tail = [&](int t) {
    if (t & 1) {  // every odd step: land the loads of steps t + 1 and t + 2, then meet
      wait_vmem();
      __syncthreads();
    }
    if (t + 1 == T) mfma_drain();
  };
  int t = 0;
  for (int si = 0; si < it.span_cnt; ++si) {
    const int len = __builtin_amdgcn_readfirstlane(sp[si].len);
    // a span may reach only the tile's keys [lo, hi) (the reference queries of one group, on a
    // tile that crosses into the next group): then every step of it is masked
    const int kr = __builtin_amdgcn_readfirstlane(sp[si].keys);
    const int klo = kr & 0xffff, khi = kr ? (kr >> 16) : kDkvKeyTile;
    const int key0 = wave * 64 + l32;
    const bool kv0 = key0 >= klo && key0 < khi, kv1 = key0 + 32 >= klo && key0 + 32 < khi;
    const int full = kr ? 0 : len / BQ;
    for (int j = 0; j < full; ++j, ++t) {
      const int b = t % NB;
      if (t + 2 < T) issue((t + 2) % NB, t + 2);
      if (active) dkv_step<D, false>(st, krow, qs[b], dos[b], rstat[b], rstat[b] + BQ, BQ, sl2);
      if (t + 2 < T) put_stat(t + 2);
      step_tail(t);
    }
    for (int off = full * BQ; off < len; off += BQ, ++t) {
      const int b = t % NB;
      if (t + 2 < T) issue((t + 2) % NB, t + 2);
      if (active)
        dkv_step<D, true>(st, krow, qs[b], dos[b], rstat[b], rstat[b] + BQ, min(BQ, len - off), sl2, kv0, kv1);
      if (t + 2 < T) put_stat(t + 2);
      step_tail(t);
    }
  }

  if (!active) return;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int r = wave * 64 + 32 * j + l32;
    if (r >= it.len) continue;
    __bf16* kout = a.dk[s] + int64_t(it.start + r) * dstride + h * D;
    __bf16* vout = a.dv[s] + int64_t(it.start + r) * dstride + h * D;
#pragma unroll
    for (int db = 0; db < ND; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 wk, wv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          wk[e] = (__bf16)(st.dk[j][db][4 * g + e] * a.scale);
          wv[e] = (__bf16)(st.dv[j][db][4 * g + e]);
        }
        *reinterpret_cast<bf16x4*>(kout + db * 32 + 8 * g + 4 * half) = wk;
        *reinterpret_cast<bf16x4*>(vout + db * 32 + 8 * g + 4 * half) = wv;
      }
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


}  // namespace sra
