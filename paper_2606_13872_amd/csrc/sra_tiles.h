// Direct global -> LDS staging of padded [rows x D] bf16 tiles and the span walk of the kernels.
#pragma once
#include "sra_config.h"
#include "sra_device.h"

namespace sra {

// Padded LDS tiles: NR rows of D bf16 with a row stride of RS elements, so every fragment
// address is one per-lane base plus a compile-time offset. The stride decides the bank
// pattern; measured on gfx950 (LDS read bytes per clock per CU, 16-byte aligned strides):
//   row stride (D = 128)   row fragment (ds_read_b128)   transpose read (ds_read_b64_tr_b16)
//   256 B                   16                            64
//   272 B  (D + 8)         128                            64
//   288 B  (D + 16)         64                           122
//   304 B  (D + 24)        128                           122
//   320 B  (D + 32)         32                           203
// so tiles read only as row fragments use D + 8, tiles read only through the transpose read
// use D + 32, and tiles read both ways use D + 24 or D + 8 with permuted rows (below).
template <int D> constexpr int kRowPadRS = D + 8;
template <int D> constexpr int kTrPadRS = D + 32;
template <int D> constexpr int kBothPadRS = D + 24;
// Tiles read both as row fragments and through the transpose read are stored at the
// row-fragment stride (D + 8) with their rows permuted inside each block of 16: logical row
// r = 4a + b (a, b < 4) sits at physical row 4b + a. A row fragment (16 consecutive rows, one
// 16-byte chunk each) still meets 16 distinct bank groups, and so does a transpose read
// (4 consecutive rows, 4 chunks each), which the plain D + 8 stride does not give. The map is
// its own inverse, and for r < 8 it sends r + 8 to perm16(r) + 2.
__host__ __device__ constexpr int perm16(int r) { return (r & ~15) | ((r & 3) << 2) | ((r >> 2) & 3); }

template <int D, int NR, int RS>
struct PaddedTile {
  static constexpr int kSlotsPerRow = RS / 8;                          // 16-byte slots per row
  static constexpr int kInstr = (NR * kSlotsPerRow + 63) / 64;         // 1 KB load instructions
  static constexpr int kElems = kInstr * 512;                          // LDS elements to reserve
};

// One GLOBAL_LOAD_LDS_DWORDX4: lane l copies 16 bytes from g to (lds + 16 l); lds is uniform.
// Issued as inline assembly on purpose: the compiler then does not see an LDS write in
// flight, and does not stall the LDS reads of the other buffers (which it cannot prove
// disjoint) until the copy lands. Every reader of a buffer filled this way waits with
// wait_vmem() and a workgroup barrier first. M0 holds the LDS address for the copy; it is
// reserved by the compiler, so it is restored right after the instruction has read it.
__device__ __forceinline__ void lds_dma_x4(const void* g, void* lds) {
  const uint32_t la = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)lds);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(g), "s"(la)
      : "memory");
}

// A wave-uniform 64-bit value held in scalar registers.
__device__ __forceinline__ uint64_t uniform_u64(uint64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(x));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(x >> 32));
  return (uint64_t(hi) << 32) | lo;
}

// LDS byte address of a __shared__ object.
template <class T>
__device__ __forceinline__ uint32_t lds_addr(const T* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// lds_dma_x4 to an LDS byte address (uniform) computed by the caller.
__device__ __forceinline__ void lds_dma_x4_at(const void* g, uint32_t la) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(g), "s"(__builtin_amdgcn_readfirstlane(la))
      : "memory");
}

// Direct global -> LDS copy (gfx950 GLOBAL_LOAD_LDS_DWORDX4) of rows [off, off + NR) of a span
// into a padded tile. Each wave instruction fills 1 KB of LDS: lane l writes the 16 bytes at
// (LDS base + 16 l), so lane l fetches the global chunk that belongs there; lanes that land on
// a pad slot fetch an in-bounds chunk that nothing reads. Rows past the span end are clamped
// to its last row (the kernels mask them). Instructions are dealt over the NW waves.
template <int D, int NR, int RS, int NW, bool kPerm = false>
__device__ __forceinline__ void tile_load_lds(__bf16* lds, const __bf16* __restrict__ src, int64_t stride,
                                              int head, int start, int len, int off, int wave) {
  using TL = PaddedTile<D, NR, RS>;
  static_assert(!kPerm || NR % 16 == 0, "permuted tiles hold whole 16-row blocks");
  constexpr int SPR = TL::kSlotsPerRow, CPR = D / 8;
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < (TL::kInstr + NW - 1) / NW; ++j) {
    const int ins = wave + j * NW;
    if (ins < TL::kInstr) {
      const int p = ins * 64 + lane;
      const int prow = min(p / SPR, NR - 1);
      const int row = kPerm ? perm16(prow) : prow;  // logical row stored at physical row prow
      const int slot = p % SPR;
      const int ch = slot < CPR ? slot : 0;
      const int rr = min(off + row, len - 1);
      const __bf16* g = src + int64_t(start + rr) * stride + head * D + ch * 8;
      lds_dma_x4(g, lds + ins * 512);
    }
  }
}

// Per-lane address offsets of the direct loads of a padded tile, for tiles whose NR rows all
// lie inside the span (no clamping): lane offsets are fixed, only the tile's first row moves.
template <int D, int NR, int RS, int NW, bool kPerm = false>
struct TileLoader {
  using TL = PaddedTile<D, NR, RS>;
  static_assert(!kPerm || NR % 16 == 0, "permuted tiles hold whole 16-row blocks");
  static constexpr int kSlots = (TL::kInstr + NW - 1) / NW;
  int voff[kSlots];  // element offset of this lane's chunk from the tile's first row
  __device__ __forceinline__ void init(int64_t stride, int head, int wave) {
    constexpr int SPR = TL::kSlotsPerRow, CPR = D / 8;
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int j = 0; j < kSlots; ++j) {
      const int p = (wave + j * NW) * 64 + lane;
      const int prow = min(p / SPR, NR - 1);
      const int row = kPerm ? perm16(prow) : prow;
      const int slot = p % SPR;
      voff[j] = int(row * stride) + head * D + (slot < CPR ? slot : 0) * 8;
    }
  }
  // `first_row` points at the tile's first row (uniform); every row is inside the span.
  __device__ __forceinline__ void issue(__bf16* lds, const __bf16* first_row, int wave) const {
#pragma unroll
    for (int j = 0; j < kSlots; ++j) {
      const int ins = wave + j * NW;
      if (ins < TL::kInstr)
        lds_dma_x4(first_row + voff[j], lds + ins * 512);
    }
  }
};

__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Walks the flattened sequence of NR-row steps over a work item's span list, keeping the
// current span's fields in registers (the span table is read once per span).
struct SpanCursor {
  const Span* spans;
  int n, si, off;
  int cur_stream, cur_start, cur_len;
  __device__ __forceinline__ void load() {
    if (si < n) {
      const Span s = spans[si];
      cur_stream = __builtin_amdgcn_readfirstlane(s.stream);
      cur_start = __builtin_amdgcn_readfirstlane(s.start);
      cur_len = __builtin_amdgcn_readfirstlane(s.len);
    }
  }
  __device__ __forceinline__ void init(const Span* s, int count) {
    spans = s;
    n = count;
    si = 0;
    off = 0;
    load();
  }
  __device__ __forceinline__ bool valid() const { return si < n; }
  __device__ __forceinline__ int stream() const { return cur_stream; }
  __device__ __forceinline__ int start() const { return cur_start; }
  __device__ __forceinline__ int len() const { return cur_len; }
  __device__ __forceinline__ void advance(int step) {
    off += step;
    if (off >= cur_len) {
      ++si;
      off = 0;
      load();
    }
  }
};

__device__ __forceinline__ int count_steps(const Span* s, int n, int step) {
  int t = 0;
  for (int i = 0; i < n; ++i) t += (s[i].len + step - 1) / step;
  return t;
}

}  // namespace sra
