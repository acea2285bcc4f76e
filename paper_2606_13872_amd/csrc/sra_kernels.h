// Kernel argument blocks and launchers (host <-> device interface inside libsra).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sra_config.h"

namespace sra {

// Streams are indexed 0 = generation, 1 = reference.
struct FwdArgs {
  const WorkItem* items;
  const Span* spans;
  const __bf16* q[2];
  const __bf16* k[2];
  const __bf16* v[2];
  int64_t in_stride[2];  // q/k/v token stride (elements) per stream
  __bf16* o[2];          // dense [rows, heads, D]
  float* lse[2];         // [heads, rows]
  int32_t rows[2];       // packed rows per stream
  int32_t heads;
  float scale_log2;      // softmax scale * log2(e)
};

struct BwdArgs {
  const WorkItem* items;
  const Span* spans;
  const __bf16* q[2];
  const __bf16* k[2];
  const __bf16* v[2];
  int64_t in_stride[2];
  const __bf16* dout[2];   // dense
  const float* lse2[2];    // [heads, rows], log-sum-exp in log2 units (written by the delta kernel)
  const float* ndelta[2];  // [heads, rows], -rowsum(dO * O)
  __bf16* dq[2];
  __bf16* dk[2];
  __bf16* dv[2];
  int32_t rows[2];
  int32_t heads;
  float scale;            // softmax scale
  float scale_log2;
};

struct DeltaArgs {
  const __bf16* o[2];
  const __bf16* dout[2];
  const float* lse[2];  // [heads, rows], natural log (the forward's output)
  float* ndelta[2];     // [heads, rows] <- -rowsum(dO * O)
  float* lse2[2];       // [heads, rows] <- lse * log2(e)
  int32_t rows[2];
  int32_t heads;
};

struct FillArgs {
  const FillRange* ranges;
  int32_t n_ranges;
  int32_t heads;
  int32_t head_dim;
  __bf16* t[3];      // dense [rows, heads, D] tensors of the range's stream to zero (may be null)
  float* lse;        // [heads, lse_rows] to set to -inf (may be null)
  int32_t lse_rows;
};

// Reference rows into the compacted stream (token masks that split frames).
constexpr int kGatherMax = 5;
struct GatherArgs {
  const int32_t* index;          // [rows]: packed ref row of each compacted row
  int32_t rows;                  // compacted rows
  int32_t row_elems;             // heads * D
  const __bf16* src[kGatherMax]; // [packed rows] tensors with token strides src_stride (may be null)
  int64_t src_stride[kGatherMax];
  __bf16* dst[kGatherMax];       // dense [rows, heads, D]
  const float* lse_src;          // [heads, lse_src_rows] (may be null)
  int32_t lse_src_rows;
  float* lse_dst;                // [heads, rows]
  int32_t heads;
};

// Compacted rows back to the packed reference stream; invalid rows get 0 (and -inf LSE).
constexpr int kScatterMax = 3;
struct ScatterArgs {
  const int32_t* index;           // [rows]: compacted row of each packed ref row, -1 = invalid
  int32_t rows;                   // packed ref rows
  int32_t row_elems;              // heads * D
  const __bf16* src[kScatterMax]; // dense [compacted rows, heads, D]
  __bf16* dst[kScatterMax];       // dense [rows, heads, D] (may be null)
  const float* lse_src;           // [heads, lse_src_rows] compacted
  int32_t lse_src_rows;
  float* lse_dst;                 // [heads, rows] (may be null)
  int32_t heads;
};

hipError_t launch_forward(const FwdArgs& a, int n_items, int head_dim, hipStream_t stream);
hipError_t launch_delta(const DeltaArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_dq(const BwdArgs& a, int n_items, int head_dim, hipStream_t stream);
hipError_t launch_dkv(const BwdArgs& a, int n_items, int head_dim, hipStream_t stream);
hipError_t launch_fill(const FillArgs& a, hipStream_t stream);
hipError_t launch_gather(const GatherArgs& a, hipStream_t stream);
hipError_t launch_scatter(const ScatterArgs& a, hipStream_t stream);

}  // namespace sra
