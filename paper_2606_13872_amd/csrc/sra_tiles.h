// Cooperative global -> register -> LDS staging of [rows x D] bf16 tiles (256 threads).
#pragma once
#include "sra_config.h"
#include "sra_device.h"

namespace sra {

template <int D, int NR>
struct TileRegs {
  static constexpr int kChunksPerRow = D / 8;  // 16-byte chunks
  static constexpr int kPerThread = NR * kChunksPerRow / kThreads;
  static_assert(kPerThread * kThreads == NR * kChunksPerRow, "tile must split evenly");
  uint4 v[kPerThread];
};

// Loads rows [off, off + NR) of the span [start, start + len) of one head. Rows past the end
// of the span are clamped to its last row, so every address stays inside the tensor; the
// kernels mask those rows out of the softmax.
template <int D, int NR>
__device__ __forceinline__ void tile_load(TileRegs<D, NR>& t, const __bf16* __restrict__ src,
                                          int64_t stride, int head, int start, int len, int off) {
  constexpr int CPR = TileRegs<D, NR>::kChunksPerRow;
#pragma unroll
  for (int i = 0; i < TileRegs<D, NR>::kPerThread; ++i) {
    const int u = int(threadIdx.x) + i * kThreads;
    const int r = u / CPR, ch = u % CPR;
    const int rr = min(off + r, len - 1);
    const __bf16* g = src + int64_t(start + rr) * stride + head * D + ch * 8;
    t.v[i] = *reinterpret_cast<const uint4*>(g);
  }
}

template <int D, int NR>
__device__ __forceinline__ void tile_store(const TileRegs<D, NR>& t, __bf16* lds) {
  constexpr int CPR = TileRegs<D, NR>::kChunksPerRow;
#pragma unroll
  for (int i = 0; i < TileRegs<D, NR>::kPerThread; ++i) {
    const int u = int(threadIdx.x) + i * kThreads;
    const int r = u / CPR, ch = u % CPR;
    *reinterpret_cast<uint4*>(lds + tile_off<D>(r, ch * 8)) = t.v[i];
  }
}

// Walks the flattened sequence of NR-row steps over a work item's span list.
struct SpanCursor {
  const Span* spans;
  int n, si, off;
  __device__ __forceinline__ void init(const Span* s, int count) { spans = s; n = count; si = 0; off = 0; }
  __device__ __forceinline__ bool valid() const { return si < n; }
  __device__ __forceinline__ int stream() const { return spans[si].stream; }
  __device__ __forceinline__ int start() const { return spans[si].start; }
  __device__ __forceinline__ int len() const { return spans[si].len; }
  __device__ __forceinline__ void advance(int step) {
    off += step;
    if (off >= spans[si].len) { ++si; off = 0; }
  }
};

__device__ __forceinline__ int count_steps(const Span* s, int n, int step) {
  int t = 0;
  for (int i = 0; i < n; ++i) t += (s[i].len + step - 1) / step;
  return t;
}

}  // namespace sra
