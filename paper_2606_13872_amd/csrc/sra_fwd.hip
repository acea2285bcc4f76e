// Forward pass of Sparse Reference Attention on gfx950.
//
// One workgroup (4 wave64s) takes one work item: a tile of up to 256 query rows of one
// stream and head, plus the list of key spans those rows see (Avatar V §1, §2.1, §4.3: gen
// rows see the gen keys and the valid ref frames of their sample; ref rows see the valid
// frames of their own group). Keys stream through LDS 64 rows at a time, double
// buffered; every wave owns 64 query rows and keeps O^T in registers:
//
//   S^T (keys x queries) = K Q^T          bf16 MFMA 32x32x16, K rows from LDS, Q^T in VGPRs
//   online softmax over keys in base 2, lanes = queries (row max/sum are lane-local plus
//   one permlane32 swap); the running max is only moved when it grows by > 8 (log2), so
//   the O rescale is rare
//   O^T (d x queries) += V^T P^T          V^T fragments via the LDS transpose read
//
// Only the last step of a span is masked (its ragged tail); there is no dense mask.
#include "sra_kernels.h"
#include "sra_tiles.h"

namespace sra {

namespace {
constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kRescaleSlack = 8.0f;  // log2 units: P may grow up to 2^8 before a rescale
}

template <int D>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
sra_fwd_kernel(FwdArgs a) {
  constexpr int NC = D / 16;  // 16-wide MFMA k-chunks over head_dim
  constexpr int ND = D / 32;  // 32-row blocks of O^T
  constexpr int BK = kFwdKeyStep;
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

  // Q^T as MFMA B fragments: lane holds query (l32) and 8 consecutive head dims.
  bf16x8 qf[2][NC];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int r = wrow0 + qb * 32 + l32;
    const __bf16* src = a.q[s] + int64_t(it.start + min(r, it.len - 1)) * a.in_stride[s] + h * D + half * 8;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      bf16x8 x = *reinterpret_cast<const bf16x8*>(src + c * 16);
      qf[qb][c] = (r < it.len) ? x : bf16x8{};
    }
  }

  floatx16 o[2][ND];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int db = 0; db < ND; ++db) o[qb][db] = floatx16{};
  float m_run[2] = {-INFINITY, -INFINITY};
  float l_part[2] = {0.f, 0.f};

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

  for (int t = 0; t < T; ++t) {
    const int buf = t & 1;
    const int nvalid = min(BK, cp.len() - cp.off);
    if (active) {
      const __bf16* kt = ks[buf];
      const __bf16* vt = vs[buf];
      floatx16 st[2][2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) st[kb][qb] = floatx16{};
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          const bf16x8 ka = *reinterpret_cast<const bf16x8*>(kt + tile_off<D>(kb * 32 + l32, c * 16 + half * 8));
#pragma unroll
          for (int qb = 0; qb < 2; ++qb) st[kb][qb] = mfma32(ka, qf[qb][c], st[kb][qb]);
        }
      if (nvalid < BK) {  // ragged end of a span
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int key = kb * 32 + 8 * (i >> 2) + 4 * half + (i & 3);
            if (key >= nvalid) {
              st[kb][0][i] = -INFINITY;
              st[kb][1][i] = -INFINITY;
            }
          }
      }
      // online softmax, base 2, lazily rescaled
      bool grow = false;
      float alpha[2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        float mx = st[0][qb][0];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int i = 0; i < 16; ++i) mx = fmaxf(mx, st[kb][qb][i]);
        mx = pair_max(mx) * sl2;
        const bool need = mx > m_run[qb] + kRescaleSlack;
        alpha[qb] = need ? fast_exp2(m_run[qb] - mx) : 1.f;
        m_run[qb] = need ? mx : m_run[qb];
        l_part[qb] *= alpha[qb];
        grow |= need;
      }
      if (__builtin_amdgcn_ballot_w64(grow) != 0) {
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
          for (int db = 0; db < ND; ++db) o[qb][db] *= alpha[qb];
      }
      bf16x8 pf[2][2][2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const float p = fast_exp2(fmaf(st[kb][qb][i], sl2, -m_run[qb]));
            st[kb][qb][i] = p;
            l_part[qb] += p;
          }
          pf[kb][qb][0] = to_bf16x8(st[kb][qb], 0);
          pf[kb][qb][1] = to_bf16x8(st[kb][qb], 8);
        }
      // O^T += V^T P^T ; V^T fragment rows = keys matching the P^T register order
      const int tcol = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
      const int trow = 4 * half + ((lane & 15) >> 2);
#pragma unroll
      for (int db = 0; db < ND; ++db)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int c2 = 0; c2 < 2; ++c2) {
            const int r0 = kb * 32 + 16 * c2 + trow;
            const bf16x4 lo = lds_read_tr(vt + tile_off<D>(r0, db * 32 + tcol));
            const bf16x4 hi = lds_read_tr(vt + tile_off<D>(r0 + 8, db * 32 + tcol));
            const bf16x8 va = cat8(lo, hi);
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) o[qb][db] = mfma32(va, pf[kb][qb][c2], o[qb][db]);
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
    const float lt = pair_sum(l_part[qb]);
    const float inv = 1.f / lt;
    const int r = wrow0 + qb * 32 + l32;
    if (r < it.len) {
      __bf16* orow = a.o[s] + int64_t(it.start + r) * ostride + h * D;
#pragma unroll
      for (int db = 0; db < ND; ++db)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          bf16x4 w;
#pragma unroll
          for (int e = 0; e < 4; ++e) w[e] = (__bf16)(o[qb][db][4 * g + e] * inv);
          *reinterpret_cast<bf16x4*>(orow + db * 32 + 8 * g + 4 * half) = w;
        }
      if (half == 0) a.lse[s][int64_t(h) * a.rows[s] + it.start + r] = (m_run[qb] + log2f(lt)) * kLn2;
    }
  }
}

hipError_t launch_forward(const FwdArgs& a, int n_items, int head_dim, hipStream_t stream) {
  if (n_items <= 0) return hipSuccess;
  if (head_dim == 128)
    hipLaunchKernelGGL(sra_fwd_kernel<128>, dim3(n_items), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(sra_fwd_kernel<64>, dim3(n_items), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace sra
