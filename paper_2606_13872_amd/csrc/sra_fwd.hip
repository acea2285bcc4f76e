// Forward pass of Sparse Reference Attention on gfx950.
//
// One workgroup (8 wave64s, two per SIMD) takes one work item: a tile of up to 256 query
// rows of one stream and head, plus the list of key spans those rows see (Avatar V §1,
// §2.1, §4.3: gen rows see the gen keys and the valid ref frames of their sample; ref rows
// see the valid frames of their own group). Every wave owns 32 query rows and keeps Q^T and
// O^T in VGPRs; keys stream through LDS in 64-row tiles (direct global->LDS loads, three
// buffers each for K and V):
//
//   S^T (keys x queries) = K Q^T          bf16 MFMA 32x32x16, K row fragments from LDS
//   online softmax over keys in base 2, lanes = queries (row sums are lane-local plus one
//   permlane32 swap)
//   O^T (d x queries) += V^T P^T          V^T fragments via the LDS transpose read
//
// The key loop is software-pipelined in 32-key halves and each wave's instruction stream is
// laid out by hand: one block issues 16 MFMAs (the P V product of the previous half and the
// S^T product of the next half), each followed by a slice of the softmax of the current
// half and by the LDS reads of the MFMA two slots ahead. A wave's MFMAs then run while the
// same wave issues its softmax arithmetic, instead of the two alternating in phases.
//
// The running max m is not tracked per half. P is computed against the current m, and its
// partial row sum doubles as the overflow check: if some lane's 16 values sum to more than
// kBigSum (some P > kBigSum, or an inf from m = -inf at the start), the wave takes the rare
// slow path: recompute that half's S, set m to the true running max, rescale O and l,
// recompute P. So m always lies within log2(kBigSum) of the true row max.
//
// Full 64-key tiles of all spans run through the pipeline first; the ragged tail of each
// span runs afterwards in a masked, unpipelined step (the accumulation is order-independent).
#include <type_traits>

#include "sra_kernels.h"
#include "sra_tiles.h"

namespace sra {

namespace {
constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kBigSum = 65536.0f;  // a lane's half-step sum of P above this forces a rescale
constexpr int kLook = 2;             // LDS fragments are read this many MFMA slots ahead
constexpr int kWaves = kFwdQueryTile / 32;
template <int D> using KTile = PaddedTile<D, kFwdKeyStep, kRowPadRS<D>>;  // row-fragment reads
template <int D> using VTile = PaddedTile<D, kFwdKeyStep, kRowPadRS<D>>;  // transpose reads, rows permuted
}  // namespace

template <int D>
struct FwdState {
  bf16x8 qf[D / 16];   // Q^T MFMA B fragments: lane = query, 8 consecutive head dims
  floatx16 o[D / 32];  // O^T accumulators, 32 head dims each
  float m;             // running max (log2 units)
  float l;             // per-lane partial row sum (fp32)
};

// P of one 32-key half for the wave's 32 query rows, as the two B fragments of the P V
// product (keys 0..15 and 16..31 of the half).
struct HalfP {
  bf16x8 p0, p1;
};

// K row fragment c of the 32 keys at kt (A operand of S^T = K Q^T).
template <int D>
__device__ __forceinline__ bf16x8 k_frag(const __bf16* kt, int c) {
  const int lane = threadIdx.x & 63;
  return *reinterpret_cast<const bf16x8*>(kt + (lane & 31) * kRowPadRS<D> + c * 16 + (lane >> 5) * 8);
}

// V^T fragment i of the 32 keys at vt (A operand of O^T += V^T P^T): i = 4*c2 + db covers
// keys 16*c2 .. 16*c2+15 and head dims 32*db .. 32*db+31. The transpose read gives lane
// (head dim) the 8 keys whose P values the B fragment holds, in the MFMA output's order.
template <int D>
__device__ __forceinline__ bf16x8 v_frag(const __bf16* vt, int i) {
  const int lane = threadIdx.x & 63;
  const int tcol = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const int trow = 4 * (lane >> 5) + ((lane & 15) >> 2);
  // rows r and r + 8 of a 16-row block sit at physical rows perm16(r) and perm16(r) + 2
  const int r0 = 16 * (i / (D / 32)) + perm16(trow), db = i % (D / 32);
  return cat8(lds_read_tr(vt + r0 * kRowPadRS<D> + db * 32 + tcol),
              lds_read_tr(vt + (r0 + 2) * kRowPadRS<D> + db * 32 + tcol));
}

// S^T of 32 keys, plain (used outside the pipeline).
template <int D>
__device__ __forceinline__ floatx16 scores32(const FwdState<D>& st, const __bf16* kt) {
  floatx16 s = floatx16{};
#pragma unroll
  for (int c = 0; c < D / 16; ++c) s = mfma32(k_frag<D>(kt, c), st.qf[c], s);
  return s;
}

// exp2(s * sl2 - m) of a half in place; returns the lane's partial sum.
__device__ __forceinline__ float exp_half(floatx16& s, float m, float sl2) {
  const float nm = -m;
  float a0 = 0.f, a1 = 0.f;
#pragma unroll
  for (int i = 0; i < 16; i += 2) {
    s[i] = fast_exp2(fmaf(s[i], sl2, nm));
    s[i + 1] = fast_exp2(fmaf(s[i + 1], sl2, nm));
    a0 += s[i];
    a1 += s[i + 1];
  }
  return a0 + a1;
}

// Rare path: s holds S^T of a half (recomputed); move m to the true running max, rescale O
// and l, and return P of the half (in s) with its partial sum.
template <int D>
__device__ __forceinline__ float rescale_half(FwdState<D>& st, floatx16& s, float sl2) {
  float mq[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) mq[j] = max3f(s[4 * j], s[4 * j + 1], max2f(s[4 * j + 2], s[4 * j + 3]));
  const float mx = pair_max(max2f(max2f(mq[0], mq[1]), max2f(mq[2], mq[3]))) * sl2;
  if (mx > st.m) {
    const float alpha = fast_exp2(st.m - mx);  // 0 when m was -inf
    st.m = mx;
    st.l *= alpha;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) st.o[db] *= alpha;
  }
  return exp_half(s, st.m, sl2);
}

// Slice J of the softmax of a half, software-pipelined over three slices so that the
// instructions issued together never depend on each other: the scale-and-shift FMA of
// elements 2 slices ahead, the exp2 of elements 1 slice ahead, and the row-sum add (and bf16
// pack) of this slice's elements. EPS elements per slice.
template <int J, int EPS>
__device__ __forceinline__ void softmax_slice(floatx16& s, float nm, float sl2, float& acc0, float& acc1,
                                              HalfP& out) {
#pragma unroll
  for (int u = 0; u < EPS; ++u) {
    constexpr int kA = (J + 2) * EPS, kB = (J + 1) * EPS, kC = J * EPS;
    if (kA + u < 16) s[kA + u] = fmaf(s[kA + u], sl2, nm);
    if (kB + u < 16) s[kB + u] = fast_exp2(s[kB + u]);
    const int e = kC + u;
    if (e & 1) {
      acc1 += s[e];
      const bf16x2 pr = {(__bf16)s[e - 1], (__bf16)s[e]};
      if (e < 8) {
        out.p0[e - 1] = pr[0];
        out.p0[e] = pr[1];
      } else {
        out.p1[e - 9] = pr[0];
        out.p1[e - 8] = pr[1];
      }
    } else {
      acc0 += s[e];
    }
  }
}

// MFMA slot pair I of a pipelined block (recursion over I = 0..NC-1): S^T MFMA I of the next
// half, then P V MFMA I of a finished half, each followed by one softmax slice of the current
// half; fragments LOOK slots ahead are read from LDS. Scheduling barriers keep the order.
template <int I, int NC, int D, int LOOK>
__device__ __forceinline__ void pipe_slots(FwdState<D>& st, floatx16& s_cur, floatx16& sn, bf16x8* kf, bf16x8* vf,
                                           const __bf16* kq, const __bf16* vp, const HalfP& pv, float nm,
                                           float sl2, float& acc0, float& acc1, HalfP& out) {
  constexpr int EPS = 16 / (2 * NC);
  if constexpr (I < NC) {
    if constexpr (I + LOOK < NC) kf[I + LOOK] = k_frag<D>(kq, I + LOOK);
    sn = mfma32(kf[I], st.qf[I], sn);
    softmax_slice<2 * I, EPS>(s_cur, nm, sl2, acc0, acc1, out);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (I + LOOK < NC) vf[I + LOOK] = v_frag<D>(vp, I + LOOK);
    constexpr int db = I % (D / 32);
    st.o[db] = mfma32(vf[I], I < D / 32 ? pv.p0 : pv.p1, st.o[db]);
    softmax_slice<2 * I + 1, EPS>(s_cur, nm, sl2, acc0, acc1, out);
    __builtin_amdgcn_sched_barrier(0);
    pipe_slots<I + 1, NC, D, LOOK>(st, s_cur, sn, kf, vf, kq, vp, pv, nm, sl2, acc0, acc1, out);
  }
}

// One pipelined block. MFMA slots alternate S^T = K Q^T of the next half (K rows at kq, into
// s_next) and O^T += V^T P^T of a finished half (V rows at vp, P in pv); after each MFMA one
// slice of the softmax of the current half (s_cur, whose K rows are at kc) is issued.
// Returns P of the current half. Slot order is fixed with scheduling barriers.
template <int D>
__device__ __forceinline__ HalfP pipe_block(FwdState<D>& st, floatx16& s_cur, const __bf16* kc,
                                            floatx16& s_next, const __bf16* kq, const __bf16* vp,
                                            const HalfP& pv, float sl2) {
  constexpr int NC = D / 16, NV = D / 16;  // QK slots, PV slots (2 key groups x D/32 dims)
  static_assert(NC == NV, "slots pair up");
  const float nm = -st.m;
  float acc0 = 0.f, acc1 = 0.f;
  HalfP out;
  bf16x8 kf[NC], vf[NV];
#pragma unroll
  for (int i = 0; i < kLook; ++i) {
    kf[i] = k_frag<D>(kq, i);
    vf[i] = v_frag<D>(vp, i);
  }
  floatx16 sn = floatx16{};
  // softmax slice j (0..2*NC-1) covers EPS elements of s_cur (1 for D = 128, 2 for D = 64)
  constexpr int EPS = 16 / (2 * NC);
  // prologue of the three-stage softmax: FMA of slices 0 and 1, exp2 of slice 0
#pragma unroll
  for (int e = 0; e < 2 * EPS; ++e) s_cur[e] = fmaf(s_cur[e], sl2, nm);
#pragma unroll
  for (int e = 0; e < EPS; ++e) s_cur[e] = fast_exp2(s_cur[e]);
  pipe_slots<0, NC, D, kLook>(st, s_cur, sn, kf, vf, kq, vp, pv, nm, sl2, acc0, acc1, out);
  s_next = sn;
  // keep the bf16 packs in the slots above (not sunk past the rare-path branch)
  asm volatile("" : "+v"(out.p0), "+v"(out.p1));
  float lsum = acc0 + acc1;
  if (__builtin_expect(__builtin_amdgcn_ballot_w64(!(lsum <= kBigSum)) != 0, 0)) {
    s_cur = scores32<D>(st, kc);
    lsum = rescale_half<D>(st, s_cur, sl2);
    out.p0 = to_bf16x8(s_cur, 0);
    out.p1 = to_bf16x8(s_cur, 8);
  }
  st.l += lsum;
  return out;
}

// O^T += V^T P^T for one half, plain.
template <int D>
__device__ __forceinline__ void pv_half(FwdState<D>& st, const __bf16* vt, const HalfP& h) {
#pragma unroll
  for (int i = 0; i < D / 16; ++i) {
    const int db = i % (D / 32);
    st.o[db] = mfma32(v_frag<D>(vt, i), i < D / 32 ? h.p0 : h.p1, st.o[db]);
  }
}

// Masked half for the ragged tails (keys >= nvalid are outside the span); always takes the
// exact path (row max, rescale when it grew), since tails are rare.
template <int D>
__device__ __forceinline__ void masked_half(FwdState<D>& st, const __bf16* kt, const __bf16* vt, int nvalid,
                                            float sl2) {
  const int half = (threadIdx.x & 63) >> 5;
  floatx16 s = scores32<D>(st, kt);
#pragma unroll
  for (int i = 0; i < 16; ++i) s[i] = (8 * (i >> 2) + 4 * half + (i & 3)) < nvalid ? s[i] : -INFINITY;
  st.l += rescale_half<D>(st, s, sl2);
  HalfP h;
  h.p0 = to_bf16x8(s, 0);
  h.p1 = to_bf16x8(s, 8);
  pv_half<D>(st, vt, h);
}

// Walks the full 64-row tiles of a span list (ragged span ends are skipped).
struct FullTileCursor {
  const Span* spans;
  int n, si, off, cur_stream, cur_start, cur_len;
  __device__ __forceinline__ void settle() {
    while (si < n) {
      const Span s = spans[si];
      cur_stream = __builtin_amdgcn_readfirstlane(s.stream);
      cur_start = __builtin_amdgcn_readfirstlane(s.start);
      cur_len = __builtin_amdgcn_readfirstlane(s.len);
      if (off + kFwdKeyStep <= cur_len) return;
      ++si;
      off = 0;
    }
  }
  __device__ __forceinline__ void init(const Span* s, int count) {
    spans = s;
    n = count;
    si = 0;
    off = 0;
    settle();
  }
  __device__ __forceinline__ void advance() {
    off += kFwdKeyStep;
    if (off + kFwdKeyStep > cur_len) {
      ++si;
      off = 0;
      settle();
    }
  }
};

template <int D>
__global__ void __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
sra_fwd_kernel(FwdArgs a) {
  constexpr int NC = D / 16, ND = D / 32, BK = kFwdKeyStep, RK = kRowPadRS<D>, RV = kRowPadRS<D>;
  constexpr int KE = KTile<D>::kElems, VE = VTile<D>::kElems;
  // Three buffers each for K and V, as separate arrays addressed only with compile-time
  // choices (the loop is unrolled by three): the compiler can then tell a buffer being filled
  // by direct loads from the ones being read, and does not stall the reads on those loads.
  __shared__ __attribute__((aligned(1024))) __bf16 kbuf0[KE];
  __shared__ __attribute__((aligned(1024))) __bf16 kbuf1[KE];
  __shared__ __attribute__((aligned(1024))) __bf16 kbuf2[KE];
  __shared__ __attribute__((aligned(1024))) __bf16 vbuf0[VE];
  __shared__ __attribute__((aligned(1024))) __bf16 vbuf1[VE];
  __shared__ __attribute__((aligned(1024))) __bf16 vbuf2[VE];
  __bf16* const kb[3] = {kbuf0, kbuf1, kbuf2};
  __bf16* const vb[3] = {vbuf0, vbuf1, vbuf2};

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
  int T = 0;  // full tiles over all spans
  for (int i = 0; i < it.span_cnt; ++i) T += __builtin_amdgcn_readfirstlane(sp[i].len) / BK;

  TileLoader<D, BK, RK, kWaves> kl[2];
  TileLoader<D, BK, RV, kWaves, true> vl[2];  // V rows permuted in blocks of 16
#pragma unroll
  for (int ss = 0; ss < 2; ++ss) {
    kl[ss].init(a.in_stride[ss], h, wave);
    vl[ss].init(a.in_stride[ss], h, wave);
  }
  FullTileCursor kc, vc;  // next full tile to load for K, for V
  kc.init(sp, it.span_cnt);
  vc.init(sp, it.span_cnt);
  // per-stream bases as uniform scalars and this wave's LDS slots as byte addresses, so a
  // tile's loads need no argument reads and no generic-to-LDS address conversions
  const uint64_t kb0 = uniform_u64(reinterpret_cast<uint64_t>(a.k[0]));
  const uint64_t kb1 = uniform_u64(reinterpret_cast<uint64_t>(a.k[1]));
  const uint64_t vb0 = uniform_u64(reinterpret_cast<uint64_t>(a.v[0]));
  const uint64_t vb1 = uniform_u64(reinterpret_cast<uint64_t>(a.v[1]));
  const int64_t st0 = a.in_stride[0], st1 = a.in_stride[1];
  using KTL = PaddedTile<D, BK, RK>;
  using VTL = PaddedTile<D, BK, RV>;
  constexpr int kKFull = KTL::kInstr / kWaves, kVFull = VTL::kInstr / kWaves;
  const bool k_extra = wave + kKFull * kWaves < KTL::kInstr;
  const bool v_extra = wave + kVFull * kWaves < VTL::kInstr;
  auto issue_k = [&](const __bf16* dst) __attribute__((always_inline)) {
    const int ss = kc.cur_stream;
    const __bf16* g = reinterpret_cast<const __bf16*>(ss ? kb1 : kb0) + int64_t(kc.cur_start + kc.off) * (ss ? st1 : st0);
    const uint32_t la = lds_addr(dst) + wave * 1024;
#pragma unroll
    for (int j = 0; j < kKFull + 1; ++j)
      if (j < kKFull || k_extra) lds_dma_x4_at(g + (ss ? kl[1].voff[j] : kl[0].voff[j]), la + j * kWaves * 1024);
    kc.advance();
  };
  auto issue_v = [&](const __bf16* dst) __attribute__((always_inline)) {
    const int ss = vc.cur_stream;
    const __bf16* g = reinterpret_cast<const __bf16*>(ss ? vb1 : vb0) + int64_t(vc.cur_start + vc.off) * (ss ? st1 : st0);
    const uint32_t la = lds_addr(dst) + wave * 1024;
#pragma unroll
    for (int j = 0; j < kVFull + 1; ++j)
      if (j < kVFull || v_extra) lds_dma_x4_at(g + (ss ? vl[1].voff[j] : vl[0].voff[j]), la + j * kWaves * 1024);
    vc.advance();
  };

  // Pipelined full tiles. Tile t sits in K buffer t % 3 and V buffer t % 3 (tile -1 in V
  // buffer 2). Iteration t reads K(t) (second half), K(t+1) (first half), V(t-1) (second
  // half) and V(t) (first half), and loads K(t+2) and V(t+1).
  if (T > 0) {
    // V buffer 2 stands for tile -1: zero its second half so the first P V (P = 0) adds 0.
    for (int e = threadIdx.x * 8; e < 32 * RV; e += kWaves * 64 * 8)
      *reinterpret_cast<bf16x8*>(vbuf2 + 32 * RV + e) = bf16x8{};
    issue_k(kbuf0);
    issue_v(vbuf0);
    if (T > 1) issue_k(kbuf1);
    wait_vmem();
    __syncthreads();
    HalfP p_hi;  // P of the previous tile's second half (zero before the first tile)
    p_hi.p0 = bf16x8{};
    p_hi.p1 = bf16x8{};
    floatx16 s_lo = floatx16{}, s_hi = floatx16{};
    if (active) s_lo = scores32<D>(st, kbuf0);
    auto iteration = [&](int t, auto phase) {
      constexpr int P = decltype(phase)::value;
      __bf16* const k_t = kb[P];
      __bf16* const k_t1 = kb[(P + 1) % 3];
      __bf16* const v_tm1 = vb[(P + 2) % 3];
      __bf16* const v_t = vb[P];
      if (t + 1 < T) issue_v(vb[(P + 1) % 3]);
      if (t + 2 < T) issue_k(kb[(P + 2) % 3]);
      if (active) {
        // block 1: S^T of this tile's second half and P V of the previous tile's second
        // half, under the softmax of this tile's first half
        const HalfP p_lo = pipe_block<D>(st, s_lo, k_t, s_hi, k_t + 32 * RK, v_tm1 + 32 * RV, p_hi, sl2);
        // block 2: S^T of the next tile's first half and P V of this tile's first half,
        // under the softmax of this tile's second half (the last iteration's S^T is unused)
        p_hi = pipe_block<D>(st, s_hi, k_t + 32 * RK, s_lo, k_t1, v_t, p_lo, sl2);
      }
      wait_vmem();
      __syncthreads();
    };
    using P0 = std::integral_constant<int, 0>;
    using P1 = std::integral_constant<int, 1>;
    using P2 = std::integral_constant<int, 2>;
    int t = 0;
    for (; t + 3 <= T; t += 3) {
      iteration(t, P0{});
      iteration(t + 1, P1{});
      iteration(t + 2, P2{});
    }
    if (t < T) iteration(t, P0{});
    if (t + 1 < T) iteration(t + 1, P1{});
    // the last tile's second half: V(T-1) sits in buffer (T-1) % 3
    if (active) {
      const int last = (T - 1) % 3;
      if (last == 0) pv_half<D>(st, vbuf0 + 32 * RV, p_hi);
      else if (last == 1) pv_half<D>(st, vbuf1 + 32 * RV, p_hi);
      else pv_half<D>(st, vbuf2 + 32 * RV, p_hi);
    }
  }

  // Ragged span tails (masked, not pipelined).
  for (int i = 0; i < it.span_cnt; ++i) {
    const Span sp_i = sp[i];
    const int len = __builtin_amdgcn_readfirstlane(sp_i.len);
    const int rem = len % BK;
    if (rem == 0) continue;
    __syncthreads();  // every wave is done with the buffers
    const int ss = __builtin_amdgcn_readfirstlane(sp_i.stream);
    const int st0 = __builtin_amdgcn_readfirstlane(sp_i.start);
    tile_load_lds<D, BK, RK, kWaves>(kbuf0, a.k[ss], a.in_stride[ss], h, st0, len, len - rem, wave);
    tile_load_lds<D, BK, RV, kWaves, true>(vbuf0, a.v[ss], a.in_stride[ss], h, st0, len, len - rem, wave);
    wait_vmem();
    __syncthreads();
    if (active) {
      masked_half<D>(st, kbuf0, vbuf0, rem, sl2);
      if (rem > 32) masked_half<D>(st, kbuf0 + 32 * RK, vbuf0 + 32 * RV, rem - 32, sl2);
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
