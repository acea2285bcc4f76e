// Tile shapes and schedule records shared by the host scheduler and the HIP kernels.
#pragma once
#include <stdint.h>

namespace sra {

// Forward: one workgroup = 8 wave64s (two per SIMD), each wave owns 32 query rows, so a work
// item covers 256 query rows; keys stream through LDS 64 at a time.
constexpr int kFwdQueryTile = 256;
constexpr int kFwdKeyStep = 64;
// dQ kernel of the backward: 256-row query tiles as in the forward, held by 4 wave64s (one per
// SIMD, 64 query rows each); keys stream through LDS 32 at a time.
constexpr int kDqQueryTile = 256;
constexpr int kDqKeyStep = 32;
// dK/dV kernel of the backward: 4 wave64s (one per SIMD) x 64 keys = 256 keys per work item;
// queries stream through LDS 32 at a time.
constexpr int kDkvKeyTile = 256;
constexpr int kDkvQueryStep = 32;

constexpr int kThreads = 256;  // block size of the element-wise kernels (delta, fill, gather, scatter)
constexpr int kNumXcd = 8;  // MI355X: 8 accelerator complex dies; workgroups go round-robin
constexpr int kCusPerXcd = 32;  // 256 compute units

// One work item: a tile of rows of one stream and head, and the list of row ranges of the
// other side it pairs with (key spans for query tiles, query spans for key tiles).
struct WorkItem {
  int32_t stream;      // 0 = generation, 1 = reference, -1 = padding (no work)
  int32_t head;
  int32_t start;       // first packed token row of the tile
  int32_t len;         // rows in the tile (<= tile size)
  int32_t span_off;    // first entry in the span table
  int32_t span_cnt;
  int32_t sample;
  int32_t reserved;
};

struct Span {
  int32_t stream;      // 0 = generation, 1 = reference
  int32_t start;       // first packed token row
  int32_t len;         // rows (> 0)
  int32_t keys;        // key-major schedules: the work item's keys [lo, hi) (tile-relative) this
                       // span reaches, packed lo | hi << 16; 0 = every key of the item
};

// Row range of a stream whose outputs are constant (invalid reference frames).
struct FillRange {
  int32_t stream;
  int32_t start;
  int32_t len;
  int32_t reserved;
};

}  // namespace sra
