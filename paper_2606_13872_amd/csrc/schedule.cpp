// Geometry -> visibility runs -> tile schedules (host).
//
// Visibility (Avatar V §1, §2.1, §4.3, §8): a gen query sees every gen key of its sample and
// every valid ref key of its sample; a valid ref query sees the valid ref keys of its own
// group of `group_frames` frames. A ref token is valid when its frame is and, if the sample
// carries a token mask, its own entry is (§4.3 invalid tokens). The rule is expressed here
// as contiguous row ranges ("spans") built from the runs of valid ref rows, so each work
// item's kernel loop visits only visible key (or query) rows and masks nothing but the
// ragged end of a span and, in the key-major schedule, the keys of a tile that a group's
// reference queries do not reach.
#include "schedule.hpp"

#include <algorithm>
#include <cmath>
#include <map>
#include <queue>
#include <cstdio>
#include <numeric>

namespace sra {

namespace {

struct Run {  // [f0, f1) frames
  int32_t f0, f1;
};

struct RowRun {  // [r0, r1) ref rows (sample-relative), all valid
  int64_t r0, r1;
};

// Maximal runs of valid ref rows inside [lo, hi).
std::vector<RowRun> valid_runs(const SampleLayout& s, int64_t lo, int64_t hi) {
  std::vector<RowRun> runs;
  for (const auto& r : s.vruns) {
    const int64_t a = std::max(lo, r.first), b = std::min(hi, r.second);
    if (a < b) runs.push_back({a, b});
  }
  return runs;
}

// Rows of ref group g0 (its first frame) of a sample.
RowRun group_rows(const SampleLayout& s, int32_t g0) {
  if (!s.gbound.empty()) return {s.gbound[g0 / s.group], s.gbound[g0 / s.group + 1]};
  return {int64_t(g0) * s.F, int64_t(std::min(s.ref_frames, g0 + s.group)) * s.F};
}

// Gen frames [f0, f1) a gen frame t sees under the sample's temporal window.
Run gen_window_frames(const SampleLayout& s, int32_t t) {
  return {std::max<int32_t>(0, t - s.window), std::min<int32_t>(s.gen_frames, t + s.window + 1)};
}

bool mul_ok(int64_t a, int64_t b, int64_t lim) { return a >= 0 && b >= 0 && (b == 0 || a <= lim / b); }

}  // namespace

sra_status make_layout(const sra_problem* p, Layout* out, std::string* err) {
  if (!p) { *err = "problem is NULL"; return SRA_ERR_INVALID_ARGUMENT; }
  if (p->batch < 1) { *err = "batch must be >= 1"; return SRA_ERR_INVALID_ARGUMENT; }
  if (p->num_heads < 1) { *err = "num_heads must be >= 1"; return SRA_ERR_INVALID_ARGUMENT; }
  if (p->head_dim != 64 && p->head_dim != 128) {
    *err = "head_dim " + std::to_string(p->head_dim) + " unsupported (64 or 128)";
    return p->head_dim > 0 ? SRA_ERR_UNSUPPORTED : SRA_ERR_INVALID_ARGUMENT;
  }
  if (!p->samples) { *err = "samples is NULL"; return SRA_ERR_INVALID_ARGUMENT; }
  if (p->flags & ~uint32_t(SRA_FLAG_GEN_QUERIES_ONLY | SRA_FLAG_GEN_WINDOW)) {
    *err = "unknown flag bits";
    return SRA_ERR_INVALID_ARGUMENT;
  }
  const bool windowed = (p->flags & SRA_FLAG_GEN_WINDOW) != 0;
  if (!(std::isfinite(p->softmax_scale))) { *err = "softmax_scale is not finite"; return SRA_ERR_INVALID_ARGUMENT; }
  const int64_t hd = int64_t(p->num_heads) * p->head_dim;
  Layout L;
  L.batch = p->batch;
  L.heads = p->num_heads;
  L.head_dim = p->head_dim;
  L.gen_only = (p->flags & SRA_FLAG_GEN_QUERIES_ONLY) != 0;
  L.scale = p->softmax_scale > 0.f ? p->softmax_scale : float(1.0 / std::sqrt(double(p->head_dim)));
  L.gen_stride = p->gen_token_stride == 0 ? hd : p->gen_token_stride;
  L.ref_stride = p->ref_token_stride == 0 ? hd : p->ref_token_stride;
  if (L.gen_stride < hd || L.ref_stride < hd) {
    *err = "token stride must be >= num_heads*head_dim";
    return SRA_ERR_INVALID_ARGUMENT;
  }
  const int64_t kRowLimit = (int64_t(1) << 31) - 1;
  // The kernels' tile loaders hold the offset of a row inside a tile (up to 63 rows past the
  // tile's first row, plus the head's columns) in 32 bits.
  if (L.gen_stride > kRowLimit / 64 || L.ref_stride > kRowLimit / 64) {
    *err = "token stride exceeds (2^31 - 1) / 64 elements (32-bit offsets inside a tile)";
    return SRA_ERR_UNSUPPORTED;
  }
  L.samples.resize(p->batch);
  for (int32_t b = 0; b < p->batch; ++b) {
    const sra_sample_geom& g = p->samples[b];
    SampleLayout& s = L.samples[b];
    const std::string tag = "sample " + std::to_string(b) + ": ";
    if (g.gen_frames < 1 || g.gen_h < 1 || g.gen_w < 1) {
      *err = tag + "generation frames/height/width must be >= 1";
      return SRA_ERR_INVALID_ARGUMENT;
    }
    if (g.ref_frames < 0 || g.ref_h < 0 || g.ref_w < 0 || (g.ref_frames > 0 && (g.ref_h < 1 || g.ref_w < 1))) {
      *err = tag + "reference frames must be >= 0 and height/width >= 1 when frames > 0";
      return SRA_ERR_INVALID_ARGUMENT;
    }
    if (g.group_frames < 1) { *err = tag + "group_frames must be >= 1"; return SRA_ERR_INVALID_ARGUMENT; }
    if (windowed && g.gen_window < 0) { *err = tag + "gen_window must be >= 0"; return SRA_ERR_INVALID_ARGUMENT; }
    if (!mul_ok(g.gen_frames, int64_t(g.gen_h) * g.gen_w, kRowLimit) ||
        !mul_ok(g.ref_frames, int64_t(g.ref_h) * g.ref_w, kRowLimit)) {
      *err = tag + "token count overflows int32";
      return SRA_ERR_INVALID_ARGUMENT;
    }
    s.G = int64_t(g.gen_frames) * g.gen_h * g.gen_w;
    s.Fg = int64_t(g.gen_h) * g.gen_w;
    s.gen_frames = g.gen_frames;
    // a window reaching every frame is no window (same schedule as full attention)
    s.window = (windowed && g.gen_window < g.gen_frames - 1) ? g.gen_window : -1;
    s.F = g.ref_frames > 0 ? int64_t(g.ref_h) * g.ref_w : 0;
    s.R = int64_t(g.ref_frames) * s.F;
    s.ref_frames = g.ref_frames;
    s.group = g.group_frames;
    // runs of valid ref rows from the frame mask and the token mask
    s.vruns.clear();
    int64_t open = -1;  // first row of the run being extended, -1 = none
    for (int32_t f = 0; f < g.ref_frames; ++f) {
      const bool fv = !g.ref_frame_valid || g.ref_frame_valid[f];
      if (!g.ref_token_valid) {  // a frame mask alone: whole frames open or close a run
        const int64_t r = int64_t(f) * s.F;
        if (fv && open < 0) open = r;
        if (!fv && open >= 0) {
          s.vruns.push_back({open, r});
          open = -1;
        }
        continue;
      }
      for (int64_t j = 0; j < s.F; ++j) {
        const int64_t r = int64_t(f) * s.F + j;
        const bool tv = fv && g.ref_token_valid[r];
        if (tv && open < 0) open = r;
        if (!tv && open >= 0) {
          s.vruns.push_back({open, r});
          open = -1;
        }
      }
    }
    if (open >= 0) s.vruns.push_back({open, s.R});
    s.gen_off = L.sum_gen;
    s.ref_off = L.sum_ref;
    L.sum_gen += s.G;
    L.sum_ref += s.R;
    if (L.sum_gen > kRowLimit || L.sum_ref > kRowLimit) {
      *err = "packed token count overflows int32";
      return SRA_ERR_INVALID_ARGUMENT;
    }
  }
  // The kernels index per-row statistics (log-sum-exp, -rowsum(dO * O)) as head * rows + row
  // and whole token rows as heads * head_dim elements, both in 32 bits.
  if (hd > kRowLimit || int64_t(L.heads) * std::max(L.sum_gen, L.sum_ref) > kRowLimit) {
    *err = "num_heads * packed tokens of a stream (or num_heads * head_dim) exceeds 2^31 - 1";
    return SRA_ERR_UNSUPPORTED;
  }
  *out = std::move(L);
  return SRA_OK;
}

void closed_form_pairs(const Layout& L, int64_t* gen_pairs, int64_t* ref_pairs) {
  int64_t gp = 0, rp = 0;
  for (const SampleLayout& s : L.samples) {
    int64_t valid_rows = 0;
    for (const auto& r : s.vruns) valid_rows += r.second - r.first;
    gp += s.G * valid_rows;
    if (s.window < 0) {
      gp += s.G * s.G;
    } else {
      for (int32_t t = 0; t < s.gen_frames; ++t) {
        const Run w = gen_window_frames(s, t);
        gp += s.Fg * s.Fg * (w.f1 - w.f0);
      }
    }
    for (int32_t g0 = 0; g0 < s.ref_frames; g0 += s.group) {
      const RowRun gr = group_rows(s, g0);
      int64_t n = 0;
      for (const RowRun& r : valid_runs(s, gr.r0, gr.r1)) n += r.r1 - r.r0;
      rp += n * n;
    }
  }
  if (gen_pairs) *gen_pairs = gp;
  if (ref_pairs) *ref_pairs = L.gen_only ? 0 : rp;
}

namespace {

struct TileClass {   // tiles sharing one span list
  int32_t stream;
  int64_t row0, rows;            // packed rows covered (tiled)
  int32_t span_off, span_cnt;
  int32_t sample;
  int64_t other_rows;            // total rows over the span list
};

// Tiles rows [row0, row0+rows) of `stream` with `tile` rows each; one item per tile and head.
void emit_items(const TileClass& c, int tile, int32_t heads, int step,
                const std::vector<Span>& spans, std::vector<std::pair<int64_t, WorkItem>>* out) {
  int64_t step_rows = 0;  // work estimate: span rows rounded up to the inner step
  for (int32_t i = 0; i < c.span_cnt; ++i) {
    int64_t l = spans[c.span_off + i].len;
    step_rows += (l + step - 1) / step * step;
  }
  for (int32_t h = 0; h < heads; ++h)
    for (int64_t r = 0; r < c.rows; r += tile) {
      WorkItem w;
      w.stream = c.stream;
      w.head = h;
      w.start = int32_t(c.row0 + r);
      w.len = int32_t(std::min<int64_t>(tile, c.rows - r));
      w.span_off = c.span_off;
      w.span_cnt = c.span_cnt;
      w.sample = c.sample;
      w.reserved = 0;
      out->push_back({int64_t(tile) * step_rows, w});
    }
}

// Orders items for launch. Workgroups are dealt round-robin over the 8 XCDs, so item k of
// the launch order runs on XCD k % 8 and each XCD consumes its own subsequence in order.
// When heads divide evenly over the XCDs, every head is pinned to one XCD (the rows it streams
// stay in that XCD's L2) and each XCD's subsequence is longest-first; otherwise the whole list
// is longest-first and the round-robin deal balances it.
// heads_in_turn: each XCD runs its heads one after another instead, each head's items
// longest-first. For key tiles, whose items are of a few similar lengths and all stream the
// head's gen queries from the first row, this keeps the workgroups resident on an XCD on one
// head and close together in its query stream (measured at 720p: half the L2 misses, 1.5 %
// faster). Query tiles keep the plain order: there the long gen tiles of all the XCD's heads
// run back to back in step, and putting each head's short ref tiles between them staggered
// the next head's start and nearly tripled the misses.
void order_items(std::vector<std::pair<int64_t, WorkItem>>& v, int32_t heads, bool heads_in_turn, Schedule* s) {
  std::stable_sort(v.begin(), v.end(), [](const auto& a, const auto& b) { return a.first > b.first; });
  s->real_items = int64_t(v.size());
  s->items.clear();
  if (heads % kNumXcd != 0 || v.empty()) {
    for (auto& e : v) s->items.push_back(e.second);
    return;
  }
  std::vector<std::vector<WorkItem>> per(kNumXcd);
  for (auto& e : v) per[e.second.head % kNumXcd].push_back(e.second);
  if (heads_in_turn)
    for (auto& q : per)
      std::stable_sort(q.begin(), q.end(), [](const WorkItem& a, const WorkItem& b) { return a.head < b.head; });
  size_t n = 0;
  for (auto& q : per) n = std::max(n, q.size());
  WorkItem pad{};
  pad.stream = -1;
  for (size_t j = 0; j < n; ++j)
    for (int x = 0; x < kNumXcd; ++x) s->items.push_back(j < per[x].size() ? per[x][j] : pad);
}

// Phase alignment of a schedule (runs after order_items with heads pinned to XCDs). The first
// span of a key tile is the sample's gen query rows, and that of a gen query tile the sample's
// gen keys: every such tile of a sample and head streams the same rows, and the tiles resident
// on an XCD share them through its L2 only while they are at nearby steps of the span at the
// same time. Tiles start whenever a compute unit frees up, so tiles of different lengths drift
// apart. Here each XCD's launch order is replayed on its compute units (one resident tile
// each, time counted in steps of the inner loop): a tile predicted to start at time t begins
// its first span at step t mod S (S = the span's steps) and wraps around, so that all tiles
// stream step t mod S at time t. The tile's pairs are unchanged (the span is cut in two); only
// the order of the sums changes, fixed by the plan.
void align_phases(int step, Schedule* s) {
  std::vector<Span> spans;
  std::map<std::pair<int32_t, int32_t>, int32_t> made;  // (span list, phase in rows) -> offset
  const size_t n = s->items.size();
  for (int x = 0; x < kNumXcd; ++x) {
    std::priority_queue<int64_t, std::vector<int64_t>, std::greater<int64_t>> free_at;
    for (int c = 0; c < kCusPerXcd; ++c) free_at.push(0);
    for (size_t k = size_t(x); k < n; k += kNumXcd) {
      WorkItem& w = s->items[k];
      if (w.stream < 0 || w.span_cnt <= 0) continue;
      const Span* l = &s->spans[size_t(w.span_off)];
      int64_t cost = 0;
      for (int32_t i = 0; i < w.span_cnt; ++i) cost += (l[i].len + step - 1) / step;
      const int64_t t0 = free_at.top();
      free_at.pop();
      free_at.push(t0 + cost);
      const int64_t first_steps = (l[0].len + step - 1) / step;
      int32_t phase = 0;
      if (l[0].stream == 0 && l[0].keys == 0 && first_steps > 1) phase = int32_t(t0 % first_steps) * step;
      const auto key = std::make_pair(w.span_off, phase);
      auto it = made.find(key);
      if (it == made.end()) {
        const int32_t off = int32_t(spans.size());
        if (phase == 0) {
          spans.push_back(l[0]);
        } else {
          spans.push_back({l[0].stream, l[0].start + phase, l[0].len - phase, 0});
          spans.push_back({l[0].stream, l[0].start, phase, 0});
        }
        spans.insert(spans.end(), l + 1, l + w.span_cnt);
        it = made.emplace(key, off).first;
      }
      w.span_cnt += phase == 0 ? 0 : 1;
      w.span_off = it->second;
    }
  }
  s->spans.swap(spans);
}

// Query-major schedule (forward and dQ): query tiles of `tile` rows, key spans per class.
void build_query_major(const Layout& L, int tile, int step, Schedule* s) {
  std::vector<TileClass> classes;
  s->spans.clear();
  for (int32_t b = 0; b < L.batch; ++b) {
    const SampleLayout& sm = L.samples[b];
    // gen queries: gen keys (all, or the frames of the temporal window) + every valid ref run.
    // With a window, query tiles are cut per gen frame so that a tile shares one key set.
    const std::vector<RowRun> ref_runs = valid_runs(sm, 0, sm.R);
    auto gen_class = [&](int64_t row0, int64_t rows, int64_t key0, int64_t keys) {
      TileClass c{0, row0, rows, int32_t(s->spans.size()), 0, b, 0};
      s->spans.push_back({0, int32_t(key0), int32_t(keys), 0});
      for (const RowRun& r : ref_runs)
        s->spans.push_back({1, int32_t(sm.ref_off + r.r0), int32_t(r.r1 - r.r0), 0});
      c.span_cnt = int32_t(s->spans.size()) - c.span_off;
      classes.push_back(c);
    };
    if (sm.window < 0) {
      gen_class(sm.gen_off, sm.G, sm.gen_off, sm.G);
    } else {
      for (int32_t t = 0; t < sm.gen_frames; ++t) {
        const Run w = gen_window_frames(sm, t);
        gen_class(sm.gen_off + t * sm.Fg, sm.Fg, sm.gen_off + w.f0 * sm.Fg, (w.f1 - w.f0) * sm.Fg);
      }
    }
    if (L.gen_only) continue;
    // ref queries: per group, keys = valid runs of the group; query tiles per valid run
    for (int32_t g0 = 0; g0 < sm.ref_frames; g0 += sm.group) {
      const RowRun gr = group_rows(sm, g0);
      std::vector<RowRun> runs = valid_runs(sm, gr.r0, gr.r1);
      if (runs.empty()) continue;
      int32_t off = int32_t(s->spans.size());
      for (const RowRun& r : runs)
        s->spans.push_back({1, int32_t(sm.ref_off + r.r0), int32_t(r.r1 - r.r0), 0});
      for (const RowRun& r : runs)
        classes.push_back({1, sm.ref_off + r.r0, r.r1 - r.r0, off, int32_t(runs.size()), b, 0});
    }
  }
  std::vector<std::pair<int64_t, WorkItem>> v;
  for (const TileClass& c : classes) emit_items(c, tile, L.heads, step, s->spans, &v);
  order_items(v, L.heads, false, s);
  if (L.heads % kNumXcd == 0) align_phases(step, s);
}

// First frame of the ref group holding sample-relative ref row r.
int32_t group_of_row(const SampleLayout& s, int64_t r) {
  if (!s.gbound.empty()) {
    const auto it = std::upper_bound(s.gbound.begin(), s.gbound.end(), r);
    return int32_t(it - s.gbound.begin() - 1) * s.group;
  }
  return int32_t(r / s.F) / s.group * s.group;
}

// Key-major schedule (dK/dV): key tiles, query spans per class.
void build_key_major(const Layout& L, int tile, int step, Schedule* s) {
  std::vector<TileClass> classes;
  std::vector<std::pair<int64_t, WorkItem>> v;
  s->spans.clear();
  std::map<std::vector<int32_t>, int32_t> lists;  // span list (flattened) -> offset
  auto intern = [&](const std::vector<Span>& l) {
    std::vector<int32_t> key;
    for (const Span& x : l) key.insert(key.end(), {x.stream, x.start, x.len, x.keys});
    auto it = lists.find(key);
    if (it != lists.end()) return it->second;
    const int32_t off = int32_t(s->spans.size());
    s->spans.insert(s->spans.end(), l.begin(), l.end());
    lists.emplace(std::move(key), off);
    return off;
  };
  for (int32_t b = 0; b < L.batch; ++b) {
    const SampleLayout& sm = L.samples[b];
    // gen keys are seen by the gen queries of the sample only (those of the frames within the
    // temporal window, if any: the window is symmetric, so key frame t' is seen from the same
    // frames that t' would see)
    if (sm.window < 0) {
      int32_t gq = int32_t(s->spans.size());
      s->spans.push_back({0, int32_t(sm.gen_off), int32_t(sm.G), 0});
      classes.push_back({0, sm.gen_off, sm.G, gq, 1, b, 0});
    } else {
      for (int32_t t = 0; t < sm.gen_frames; ++t) {
        const Run w = gen_window_frames(sm, t);
        int32_t gq = int32_t(s->spans.size());
        s->spans.push_back({0, int32_t(sm.gen_off + w.f0 * sm.Fg), int32_t((w.f1 - w.f0) * sm.Fg), 0});
        classes.push_back({0, sm.gen_off + t * sm.Fg, sm.Fg, gq, 1, b, 0});
      }
    }
    // valid ref keys are seen by every gen query of the sample and by the valid ref queries of
    // their group. Tiles run across group boundaries inside each run of valid rows (a group's
    // last tile would otherwise be mostly empty and still stream every gen query); a tile's
    // span for one group's ref queries carries the range of the tile's keys in that group.
    for (const auto& run : sm.vruns) {
      for (int64_t a = run.first; a < run.second; a += tile) {
        const int64_t e = std::min<int64_t>(a + tile, run.second);
        std::vector<Span> l{{0, int32_t(sm.gen_off), int32_t(sm.G), 0}};
        if (!L.gen_only) {
          for (int32_t g0 = group_of_row(sm, a); g0 < sm.ref_frames; g0 += sm.group) {
            const RowRun gr = group_rows(sm, g0);
            if (gr.r0 >= e) break;
            const int64_t lo = std::max(a, gr.r0), hi = std::min(e, gr.r1);
            if (lo >= hi) continue;
            const int32_t keys = (lo == a && hi == e) ? 0 : int32_t(((hi - a) << 16) | (lo - a));
            for (const RowRun& q : valid_runs(sm, gr.r0, gr.r1))
              l.push_back({1, int32_t(sm.ref_off + q.r0), int32_t(q.r1 - q.r0), keys});
          }
        }
        const int32_t off = intern(l);
        int64_t step_rows = 0;
        for (const Span& x : l) step_rows += (x.len + step - 1) / step * step;
        for (int32_t h = 0; h < L.heads; ++h) {
          WorkItem w;
          w.stream = 1;
          w.head = h;
          w.start = int32_t(sm.ref_off + a);
          w.len = int32_t(e - a);
          w.span_off = off;
          w.span_cnt = int32_t(l.size());
          w.sample = b;
          w.reserved = 0;
          v.push_back({int64_t(tile) * step_rows, w});
        }
      }
    }
  }
  for (const TileClass& c : classes) emit_items(c, tile, L.heads, step, s->spans, &v);
  order_items(v, L.heads, true, s);
  if (L.heads % kNumXcd == 0) align_phases(step, s);
}

}  // namespace

bool needs_compaction(const Layout& L) {
  for (const SampleLayout& s : L.samples) {
    int64_t groups = 0;
    for (int32_t g0 = 0; g0 < s.ref_frames; g0 += s.group) {
      const RowRun gr = group_rows(s, g0);
      if (!valid_runs(s, gr.r0, gr.r1).empty()) ++groups;
    }
    if (int64_t(s.vruns.size()) > groups) return true;
  }
  return false;
}

void compact_layout(const Layout& L, Layout* C, std::vector<int32_t>* gather, std::vector<int32_t>* scatter) {
  *C = L;
  C->sum_ref = 0;
  gather->clear();
  scatter->assign(size_t(L.sum_ref), -1);
  for (size_t b = 0; b < L.samples.size(); ++b) {
    const SampleLayout& s = L.samples[b];
    SampleLayout& c = C->samples[b];
    c.ref_off = C->sum_ref;
    c.gbound.assign(1, 0);
    int64_t n = 0;
    for (int32_t g0 = 0; g0 < s.ref_frames; g0 += s.group) {
      const RowRun gr = group_rows(s, g0);
      for (const RowRun& r : valid_runs(s, gr.r0, gr.r1))
        for (int64_t row = r.r0; row < r.r1; ++row, ++n) {
          (*scatter)[size_t(s.ref_off + row)] = int32_t(c.ref_off + n);
          gather->push_back(int32_t(s.ref_off + row));
        }
      c.gbound.push_back(n);
    }
    c.R = n;
    c.vruns.clear();
    if (n > 0) c.vruns.push_back({0, n});
    C->sum_ref += n;
  }
}

void build_plan(const Layout& L_in, Plan* plan) {
  plan->layout = L_in;
  plan->compacted = needs_compaction(L_in);
  plan->ref_gather.clear();
  plan->ref_scatter.clear();
  if (plan->compacted)
    compact_layout(L_in, &plan->exec, &plan->ref_gather, &plan->ref_scatter);
  else
    plan->exec = L_in;
  const Layout& L = plan->exec;
  build_query_major(L, kFwdQueryTile, kFwdKeyStep, &plan->fwd);
  build_query_major(L, kDqQueryTile, kDqKeyStep, &plan->dq);
  build_key_major(L, kDkvKeyTile, kDkvQueryStep, &plan->dkv);
  plan->fill.clear();
  for (const SampleLayout& sm : L.samples) {  // the gaps between valid ref runs
    int64_t r = 0;
    for (const auto& v : sm.vruns) {
      if (v.first > r) plan->fill.push_back({1, int32_t(sm.ref_off + r), int32_t(v.first - r), 0});
      r = v.second;
    }
    if (r < sm.R) plan->fill.push_back({1, int32_t(sm.ref_off + r), int32_t(sm.R - r), 0});
  }
}

int64_t covered_pairs(const Schedule& s, bool /*key_major*/) {
  int64_t n = 0;
  for (const WorkItem& w : s.items) {
    if (w.stream < 0 || w.head != 0) continue;
    for (int32_t i = 0; i < w.span_cnt; ++i) {
      const Span& x = s.spans[w.span_off + i];
      const int64_t keys = x.keys ? (x.keys >> 16) - (x.keys & 0xffff) : w.len;
      n += keys * x.len;
    }
  }
  return n;
}

std::string layout_key(const Layout& L) {
  std::string k;
  auto put = [&k](int64_t v) { k.append(reinterpret_cast<const char*>(&v), sizeof v); };
  put(L.batch); put(L.heads); put(L.head_dim); put(L.gen_only ? 1 : 0);
  for (const SampleLayout& s : L.samples) {
    put(s.G); put(s.R); put(s.F); put(s.Fg); put(s.ref_frames); put(s.group); put(s.window);
    put(int64_t(s.vruns.size()));
    for (const auto& r : s.vruns) { put(r.first); put(r.second); }
  }
  return k;
}

}  // namespace sra
