// Host-side geometry validation and tile scheduling for Sparse Reference Attention.
// Pure C++ (no HIP): turns per-sample frame geometry into work-item tables.
#pragma once
#include <stdint.h>

#include <string>
#include <utility>
#include <vector>

#include "sra.h"
#include "sra_config.h"

namespace sra {

// Derived geometry of one sample.
struct SampleLayout {
  int64_t G = 0, R = 0, F = 0;        // gen tokens, ref tokens, tokens per ref frame
  int64_t Fg = 0;                     // tokens per gen frame
  int64_t gen_off = 0, ref_off = 0;   // first packed row of the sample in each stream
  int32_t gen_frames = 0, ref_frames = 0, group = 1;
  int32_t window = -1;                // gen-gen temporal window in frames; -1 = none
  // maximal runs [first, last) of valid ref token rows (sample-relative): a token is valid when
  // its frame is and, with a token mask, its own entry is
  std::vector<std::pair<int64_t, int64_t>> vruns;
  // Row bounds of the ref groups when they are not runs of F-row frames (the compacted
  // reference stream, below): group i holds rows [gbound[i], gbound[i + 1]). Empty otherwise.
  std::vector<int64_t> gbound;
};

struct Layout {
  int32_t batch = 0, heads = 0, head_dim = 0;
  float scale = 0.f;
  int64_t gen_stride = 0, ref_stride = 0;  // q/k/v token strides (elements)
  int64_t sum_gen = 0, sum_ref = 0;
  bool gen_only = false;                   // SRA_FLAG_GEN_QUERIES_ONLY: no reference queries
  std::vector<SampleLayout> samples;
};

// A schedule: work items (already in launch order, padded for the XCD mapping) and spans.
struct Schedule {
  std::vector<WorkItem> items;
  std::vector<Span> spans;
  int64_t real_items = 0;
};

// When a token mask splits reference frames into many short runs of valid tokens, tiles cut
// per run would be mostly empty. Such a plan runs on the compacted reference stream instead:
// the valid ref tokens of the batch gathered back to back (sample-major, then group-major,
// keeping their order), so every group is one contiguous run. The library gathers the
// reference inputs into that stream before the kernels and scatters the outputs back after.
struct Plan {
  Layout layout;                   // as given
  bool compacted = false;          // the schedules index the compacted reference stream
  Layout exec;                     // the layout the schedules index (layout, or its compaction)
  Schedule fwd, dq, dkv;
  std::vector<FillRange> fill;     // invalid reference rows of exec (none when compacted)
  std::vector<int32_t> ref_gather;   // compacted: packed ref row of each compacted row
  std::vector<int32_t> ref_scatter;  // compacted: compacted row of each packed ref row, or -1
};

// Validates `p` and derives the layout. Returns SRA_OK or an error with `err` set.
sra_status make_layout(const sra_problem* p, Layout* out, std::string* err);

// Closed-form visible pairs per head (summed over samples).
void closed_form_pairs(const Layout& L, int64_t* gen_pairs, int64_t* ref_pairs);

// True when some sample's token mask splits its reference frames into more runs of valid
// tokens than it has groups with a valid token (frame masks alone never do).
bool needs_compaction(const Layout& L);

// The compacted form of L (every sample's valid ref tokens back to back, groups given by
// gbound) with the row maps between the two reference streams.
void compact_layout(const Layout& L, Layout* C, std::vector<int32_t>* gather, std::vector<int32_t>* scatter);

// Builds the three schedules and the fill list (on the compacted layout when needed).
void build_plan(const Layout& L, Plan* plan);

// Pairs per head covered by a schedule (head 0 items only, so per head).
int64_t covered_pairs(const Schedule& s, bool key_major);

// Geometry key for the plan cache.
std::string layout_key(const Layout& L);

}  // namespace sra
