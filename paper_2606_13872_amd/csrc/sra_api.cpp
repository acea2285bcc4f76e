// C ABI of libsra (include/sra.h): validation, plan cache, workspace layout and launches.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <list>
#include <memory>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include "sra.h"
#include "schedule.hpp"
#include "sra_kernels.h"
#include "sra_internal.h"

namespace {

using namespace sra;

thread_local std::string g_last_error;

sra_status fail(sra_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Pinned host staging buffer for uploading a plan's tables, with the events recorded after the
// copies enqueued out of it. A buffer is reused for another plan once every such copy has run
// (checked with hipEventQuery, never by waiting), so evicting a plan neither synchronises nor
// frees anything; buffers are freed only by sra_release_caches.
struct Staging {
  void* ptr = nullptr;
  size_t bytes = 0;
  const void* owner = nullptr;     // the Blob whose image the buffer holds (nullptr = retired)
  std::vector<hipEvent_t> pending; // one per enqueued copy not yet known to be complete
};

// Byte image of a set of tables, laid out back to back (each 256-byte aligned). The pinned
// copy is made on first upload, so sizes can be queried without a device.
struct Blob {
  std::vector<size_t> offsets;
  std::vector<char> image;
  size_t bytes = 0;
  Staging* stage = nullptr;        // owned by the plan cache; valid while stage->owner == this
};

struct CachedPlan {
  Plan plan;
  uint64_t id = 0;  // unique per plan built by this process
  Blob fwd;   // fwd items | fwd spans | fill | ref gather | ref scatter
  Blob bwd;   // dq items | dq spans | dkv items | dkv spans | fill | ref gather | ref scatter
};

template <class T>
void put_table(Blob& b, const std::vector<T>& v) {
  size_t off = align_up(b.image.size());
  b.image.resize(off + v.size() * sizeof(T));
  if (!v.empty()) std::memcpy(b.image.data() + off, v.data(), v.size() * sizeof(T));
  b.offsets.push_back(off);
  b.bytes = align_up(b.image.size());
}

class PlanCache {
 public:

  sra_status get(const Layout& L, std::shared_ptr<CachedPlan>* out) {
    std::lock_guard<std::mutex> lk(mu_);
    std::string key = layout_key(L);
    auto it = map_.find(key);
    if (it != map_.end()) {
      lru_.splice(lru_.begin(), lru_, it->second.second);
      *out = it->second.first;
      return SRA_OK;
    }
    auto cp = std::make_shared<CachedPlan>();
    build_plan(L, &cp->plan);
    cp->id = ++next_id_;
    put_table(cp->fwd, cp->plan.fwd.items);
    put_table(cp->fwd, cp->plan.fwd.spans);
    put_table(cp->fwd, cp->plan.fill);
    put_table(cp->fwd, cp->plan.ref_gather);
    put_table(cp->fwd, cp->plan.ref_scatter);
    put_table(cp->bwd, cp->plan.dq.items);
    put_table(cp->bwd, cp->plan.dq.spans);
    put_table(cp->bwd, cp->plan.dkv.items);
    put_table(cp->bwd, cp->plan.dkv.spans);
    put_table(cp->bwd, cp->plan.fill);
    put_table(cp->bwd, cp->plan.ref_gather);
    put_table(cp->bwd, cp->plan.ref_scatter);
    if (map_.size() >= kMaxPlans) evict_one();
    lru_.push_front(key);
    map_[key] = {cp, lru_.begin()};
    *out = cp;
    return SRA_OK;
  }

  // Enqueues the copy of blob `b` into device memory `dst` on `s` (from its pinned staging
  // buffer, filled on first use) and records an event after it.
  sra_status upload(Blob& b, void* dst, hipStream_t s) {
    if (!b.bytes) return SRA_OK;
    std::lock_guard<std::mutex> lk(mu_);
    if (!b.stage || b.stage->owner != &b) {
      sra_status st = acquire(b);
      if (st != SRA_OK) return st;
    }
    Staging& g = *b.stage;
    hipError_t e = hipMemcpyAsync(dst, g.ptr, b.bytes, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return fail(SRA_ERR_HIP, std::string("schedule upload: ") + hipGetErrorString(e));
    hipEvent_t ev = nullptr;
    if (!free_events_.empty()) {
      ev = free_events_.back();
      free_events_.pop_back();
    } else if ((e = hipEventCreateWithFlags(&ev, hipEventDisableTiming)) != hipSuccess) {
      return fail(SRA_ERR_HIP, std::string("event for the schedule upload: ") + hipGetErrorString(e));
    }
    if ((e = hipEventRecord(ev, s)) != hipSuccess) {
      free_events_.push_back(ev);
      return fail(SRA_ERR_HIP, std::string("event after the schedule upload: ") + hipGetErrorString(e));
    }
    g.pending.push_back(ev);
    return SRA_OK;
  }

  // Waits for every upload, then frees the staging buffers and drops every plan (calls still
  // holding a plan re-stage its image on their next upload).
  void clear() {
    std::lock_guard<std::mutex> lk(mu_);
    for (auto& g : stagings_) {
      for (hipEvent_t ev : g->pending) {
        (void)hipEventSynchronize(ev);
        (void)hipEventDestroy(ev);
      }
      if (g->ptr) (void)hipHostFree(g->ptr);
    }
    stagings_.clear();
    for (hipEvent_t ev : free_events_) (void)hipEventDestroy(ev);
    free_events_.clear();
    map_.clear();
    lru_.clear();
  }

  size_t staging_buffers() {
    std::lock_guard<std::mutex> lk(mu_);
    return stagings_.size();
  }

 private:
  static constexpr size_t kMaxPlans = 256;

  // Moves the completed events of `g` to the free list; true when none is pending.
  bool reap(Staging& g) {
    size_t keep = 0;
    bool not_ready = false;
    for (hipEvent_t ev : g.pending) {
      const hipError_t q = hipEventQuery(ev);
      if (q == hipSuccess) {
        free_events_.push_back(ev);
      } else {
        g.pending[keep++] = ev;
        not_ready |= q == hipErrorNotReady;
      }
    }
    g.pending.resize(keep);
    if (not_ready) (void)hipGetLastError();  // a copy still running is not an error of any call
    return keep == 0;
  }

  // Gives blob `b` a staging buffer holding its image: a retired one that is large enough and
  // no longer read by any copy, else a new pinned allocation.
  sra_status acquire(Blob& b) {
    Staging* pick = nullptr;
    for (auto& g : stagings_)
      if (!g->owner && g->bytes >= b.bytes && reap(*g) && (!pick || g->bytes < pick->bytes)) pick = g.get();
    if (!pick) {
      void* p = nullptr;
      if (hipHostMalloc(&p, b.bytes, hipHostMallocDefault) != hipSuccess) {
        (void)hipGetLastError();
        return fail(SRA_ERR_HIP, "hipHostMalloc of schedule staging failed");
      }
      stagings_.push_back(std::make_unique<Staging>());
      pick = stagings_.back().get();
      pick->ptr = p;
      pick->bytes = b.bytes;
    }
    std::memcpy(pick->ptr, b.image.data(), b.image.size());
    pick->owner = &b;
    b.stage = pick;
    return SRA_OK;
  }

  void retire(Blob& b) {
    if (b.stage && b.stage->owner == &b) b.stage->owner = nullptr;
  }

  void evict_one() {
    auto it = map_.find(lru_.back());
    retire(it->second.first->fwd);
    retire(it->second.first->bwd);
    map_.erase(it);
    lru_.pop_back();
  }
  std::mutex mu_;
  std::list<std::string> lru_;
  std::unordered_map<std::string, std::pair<std::shared_ptr<CachedPlan>, std::list<std::string>::iterator>> map_;
  std::vector<std::unique_ptr<Staging>> stagings_;
  std::vector<hipEvent_t> free_events_;
  uint64_t next_id_ = 0;
};

PlanCache& cache() {
  static PlanCache* c = new PlanCache();  // never destroyed: HIP may be torn down first at exit
  return *c;
}

// Schedules resident in the static scratch of each device (the allocation-free forward). The
// scratch keeps the last call's tables, so a call with the plan and stream of the previous
// call on that device skips the upload; any other call copies the tables from the plan's host
// image (pageable memory, so no pinned staging is allocated).
class ResidentTables {
 public:
  sra_status upload(const Blob& b, uint64_t plan_id, int device, void* dst, hipStream_t s) {
    std::lock_guard<std::mutex> lk(mu_);
    Entry& e = by_device_[device];
    if (e.plan_id == plan_id && e.stream == s) return SRA_OK;
    e.plan_id = 0;
    if (!b.image.empty()) {
      hipError_t r = hipMemcpyAsync(dst, b.image.data(), b.image.size(), hipMemcpyHostToDevice, s);
      if (r != hipSuccess) return fail(SRA_ERR_HIP, std::string("schedule upload: ") + hipGetErrorString(r));
    }
    e.plan_id = plan_id;
    e.stream = s;
    return SRA_OK;
  }
  void clear() {
    std::lock_guard<std::mutex> lk(mu_);
    by_device_.clear();
  }

 private:
  struct Entry {
    uint64_t plan_id = 0;
    hipStream_t stream = nullptr;
  };
  std::mutex mu_;
  std::unordered_map<int, Entry> by_device_;
};

ResidentTables& resident() {
  static ResidentTables* r = new ResidentTables();
  return *r;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// Bytes of `rows` dense bf16 rows of all heads, and of one fp32 value per (head, row).
size_t rows_bytes(const Layout& L, int64_t rows) { return align_up(size_t(rows) * L.heads * L.head_dim * 2); }
size_t stat_bytes(const Layout& L, int64_t rows) { return align_up(size_t(L.heads) * rows * sizeof(float)); }

// Forward workspace: schedule, then (compacted plans) the compacted ref q, k, v, o and lse.
size_t fwd_workspace(const CachedPlan& cp) {
  const Layout& E = cp.plan.exec;
  size_t b = cp.fwd.bytes;
  if (cp.plan.compacted) b += 4 * rows_bytes(E, E.sum_ref) + stat_bytes(E, E.sum_ref);
  return b;
}
// Backward workspace: schedule; -D and the LSE in log2 units per query row of each stream;
// then (compacted plans) the compacted ref q, k, v, o, do, dq, dk, dv and lse.
size_t bwd_workspace(const CachedPlan& cp) {
  const Layout& E = cp.plan.exec;
  size_t b = cp.bwd.bytes + 2 * stat_bytes(E, E.sum_gen) + 2 * stat_bytes(E, E.sum_ref);
  if (cp.plan.compacted) b += 8 * rows_bytes(E, E.sum_ref) + stat_bytes(E, E.sum_ref);
  return b;
}

sra_status common_checks(const sra_problem* p, Layout* L, std::shared_ptr<CachedPlan>* cp) {
  std::string err;
  sra_status st = make_layout(p, L, &err);
  if (st != SRA_OK) return fail(st, err);
  if (L->gen_stride % 8 || L->ref_stride % 8)
    return fail(SRA_ERR_INVALID_ARGUMENT, "token strides must be multiples of 8 elements");
  st = cache().get(*L, cp);
  return st;
}

sra_status check_tensors(const Layout& L, std::initializer_list<const void*> gen,
                         std::initializer_list<const void*> ref) {
  for (const void* t : gen) {
    if (!t) return fail(SRA_ERR_INVALID_ARGUMENT, "a generation tensor pointer is NULL");
    if (!aligned16(t)) return fail(SRA_ERR_INVALID_ARGUMENT, "tensor pointers must be 16-byte aligned");
  }
  if (L.sum_ref > 0)
    for (const void* t : ref) {
      if (!t) return fail(SRA_ERR_INVALID_ARGUMENT, "a reference tensor pointer is NULL");
      if (!aligned16(t)) return fail(SRA_ERR_INVALID_ARGUMENT, "tensor pointers must be 16-byte aligned");
    }
  return SRA_OK;
}

sra_status hip_fail(hipError_t e, const char* what) {
  return fail(SRA_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Opt-in per-kernel timing: launches are bracketed by events on the launch stream; the
// elapsed times are collected when read.
class KernelTimer {
 public:
  void enable(bool on) {
    std::lock_guard<std::mutex> lk(mu_);
    drain();
    for (auto& ev : pending_) destroy(ev);
    pending_.clear();
    for (int i = 0; i < SRA_KERNEL_COUNT; ++i) total_[i] = 0.0, count_[i] = 0;
    on_ = on;
  }
  bool on() const { return on_; }
  // Returns an event recorded on `s` (nullptr if timing is off or the event failed).
  hipEvent_t mark(hipStream_t s) {
    if (!on_) return nullptr;
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    if (hipEventRecord(e, s) != hipSuccess) {
      (void)hipEventDestroy(e);
      return nullptr;
    }
    return e;
  }
  void add(int kernel, hipEvent_t a, hipEvent_t b) {
    if (!a || !b) {
      if (a) (void)hipEventDestroy(a);
      if (b) (void)hipEventDestroy(b);
      return;
    }
    std::lock_guard<std::mutex> lk(mu_);
    pending_.push_back({kernel, a, b});
  }
  void read(int kernel, double* ms, int64_t* n) {
    std::lock_guard<std::mutex> lk(mu_);
    drain();
    if (ms) *ms = total_[kernel];
    if (n) *n = count_[kernel];
  }

 private:
  struct Ev { int k; hipEvent_t a, b; };
  static void destroy(Ev& e) {
    (void)hipEventDestroy(e.a);
    (void)hipEventDestroy(e.b);
  }
  void drain() {
    for (auto& e : pending_) {
      float t = 0.f;
      if (hipEventSynchronize(e.b) == hipSuccess && hipEventElapsedTime(&t, e.a, e.b) == hipSuccess) {
        total_[e.k] += t;
        count_[e.k] += 1;
      }
      destroy(e);
    }
    pending_.clear();
  }
  std::mutex mu_;
  bool on_ = false;
  std::vector<Ev> pending_;
  double total_[SRA_KERNEL_COUNT] = {};
  int64_t count_[SRA_KERNEL_COUNT] = {};
};

KernelTimer& timer() {
  static KernelTimer* t = new KernelTimer();
  return *t;
}

// Launches `fn` (returning hipError_t) with optional timing under kernel id `k`.
template <class Fn>
hipError_t timed(int k, hipStream_t s, Fn&& fn) {
  hipEvent_t a = timer().mark(s);
  hipError_t e = fn();
  hipEvent_t b = timer().mark(s);
  timer().add(k, a, b);
  return e;
}

}  // namespace

extern "C" {

sra_status sra_workspace_size(const sra_problem* p, int backward, size_t* bytes) {
  g_last_error.clear();
  if (!bytes) return fail(SRA_ERR_INVALID_ARGUMENT, "bytes is NULL");
  Layout L;
  std::shared_ptr<CachedPlan> cp;
  sra_status st = common_checks(p, &L, &cp);
  if (st != SRA_OK) return st;
  *bytes = backward ? bwd_workspace(*cp) : fwd_workspace(*cp);
  return SRA_OK;
}

}  // extern "C"

namespace sra {

sra_status forward_call(const sra_problem* p, const void* q_gen, const void* k_gen, const void* v_gen,
                        const void* q_ref, const void* k_ref, const void* v_ref, void* o_gen, void* o_ref,
                        float* lse_gen, float* lse_ref, void* workspace, size_t workspace_bytes, void* stream,
                        StaticWorkspaceFn static_ws, size_t static_bytes) {
  g_last_error.clear();
  Layout L;
  std::shared_ptr<CachedPlan> cp;
  sra_status st = common_checks(p, &L, &cp);
  if (st != SRA_OK) return st;
  st = L.gen_only ? check_tensors(L, {q_gen, k_gen, v_gen, o_gen, lse_gen}, {k_ref, v_ref})
                  : check_tensors(L, {q_gen, k_gen, v_gen, o_gen, lse_gen}, {q_ref, k_ref, v_ref, o_ref, lse_ref});
  if (st != SRA_OK) return st;
  const size_t need = fwd_workspace(*cp);
  StaticWorkspace sws{nullptr, 0, -1};
  const StaticWorkspace* sw = nullptr;
  if (static_ws) {
    if (need > static_bytes)
      return fail(SRA_ERR_WORKSPACE_TOO_SMALL, "forward needs " + std::to_string(need) +
                                                   " workspace bytes, more than the static scratch maximum of " +
                                                   std::to_string(static_bytes) + " (use sra_forward)");
    st = static_ws(stream, &sws);
    if (st != SRA_OK) return st;
    if (!sws.ptr) return fail(SRA_ERR_INTERNAL, "static scratch has no device address");
    sw = &sws;
    workspace = sws.ptr;
    workspace_bytes = sws.bytes;
  }
  if (workspace_bytes < need)
    return fail(SRA_ERR_WORKSPACE_TOO_SMALL, "forward needs " + std::to_string(need) + " workspace bytes");
  if (need && (!workspace || (reinterpret_cast<uintptr_t>(workspace) % kAlign)))
    return fail(SRA_ERR_INVALID_ARGUMENT, "workspace must be non-NULL and 256-byte aligned");

  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  if (sw) st = resident().upload(cp->fwd, cp->id, sw->device, ws, s);
  else st = cache().upload(cp->fwd, ws, s);
  if (st != SRA_OK) return st;
  const Plan& P = cp->plan;
  const Layout& E = P.exec;
  const int32_t row_elems = L.heads * L.head_dim;
  FwdArgs a{};
  a.items = reinterpret_cast<const WorkItem*>(ws + cp->fwd.offsets[0]);
  a.spans = reinterpret_cast<const Span*>(ws + cp->fwd.offsets[1]);
  a.q[0] = static_cast<const __bf16*>(q_gen);
  a.k[0] = static_cast<const __bf16*>(k_gen);
  a.v[0] = static_cast<const __bf16*>(v_gen);
  a.q[1] = static_cast<const __bf16*>(q_ref);
  a.k[1] = static_cast<const __bf16*>(k_ref);
  a.v[1] = static_cast<const __bf16*>(v_ref);
  a.in_stride[0] = L.gen_stride;
  a.in_stride[1] = L.ref_stride;
  a.o[0] = static_cast<__bf16*>(o_gen);
  a.o[1] = static_cast<__bf16*>(o_ref);
  a.lse[0] = lse_gen;
  a.lse[1] = lse_ref;
  a.rows[0] = int32_t(L.sum_gen);
  a.rows[1] = int32_t(E.sum_ref);
  a.heads = L.heads;
  a.scale_log2 = float(double(L.scale) * 1.4426950408889634);
  hipError_t e;
  __bf16* o_c = nullptr;
  float* lse_c = nullptr;
  if (P.compacted) {  // the kernels read and write the compacted reference stream
    char* c = ws + cp->fwd.bytes;
    const size_t rb = rows_bytes(E, E.sum_ref);
    __bf16* qkv_c[3] = {reinterpret_cast<__bf16*>(c), reinterpret_cast<__bf16*>(c + rb),
                        reinterpret_cast<__bf16*>(c + 2 * rb)};
    o_c = reinterpret_cast<__bf16*>(c + 3 * rb);
    lse_c = reinterpret_cast<float*>(c + 4 * rb);
    GatherArgs g{};
    g.index = reinterpret_cast<const int32_t*>(ws + cp->fwd.offsets[3]);
    g.rows = int32_t(E.sum_ref);
    g.row_elems = row_elems;
    g.heads = L.heads;
    g.src[0] = L.gen_only ? nullptr : a.q[1];  // no reference queries when gen-only
    g.src[1] = a.k[1];
    g.src[2] = a.v[1];
    for (int t = 0; t < 3; ++t) {
      g.src_stride[t] = L.ref_stride;
      g.dst[t] = qkv_c[t];
    }
    e = timed(SRA_KERNEL_GATHER, s, [&] { return launch_gather(g, s); });
    if (e != hipSuccess) return hip_fail(e, "gather launch");
    a.q[1] = L.gen_only ? nullptr : qkv_c[0];
    a.k[1] = qkv_c[1];
    a.v[1] = qkv_c[2];
    a.in_stride[1] = row_elems;
    a.o[1] = o_c;
    a.lse[1] = lse_c;
  }
  e = timed(SRA_KERNEL_FORWARD, s, [&] { return launch_forward(a, int(P.fwd.items.size()), L.head_dim, s); });
  if (e != hipSuccess) return hip_fail(e, "forward launch");
  if (P.compacted && !L.gen_only) {
    ScatterArgs sc{};
    sc.index = reinterpret_cast<const int32_t*>(ws + cp->fwd.offsets[4]);
    sc.rows = int32_t(L.sum_ref);
    sc.row_elems = row_elems;
    sc.heads = L.heads;
    sc.src[0] = o_c;
    sc.dst[0] = static_cast<__bf16*>(o_ref);
    sc.lse_src = lse_c;
    sc.lse_src_rows = int32_t(E.sum_ref);
    sc.lse_dst = lse_ref;
    e = timed(SRA_KERNEL_SCATTER, s, [&] { return launch_scatter(sc, s); });
    if (e != hipSuccess) return hip_fail(e, "scatter launch");
  }
  if (!P.fill.empty() && !L.gen_only) {  // ref rows of invalid frames (no ref rows when gen-only)
    FillArgs f{};
    f.ranges = reinterpret_cast<const FillRange*>(ws + cp->fwd.offsets[2]);
    f.n_ranges = int32_t(P.fill.size());
    f.heads = L.heads;
    f.head_dim = L.head_dim;
    f.t[0] = static_cast<__bf16*>(o_ref);
    f.lse = lse_ref;
    f.lse_rows = int32_t(L.sum_ref);
    e = timed(SRA_KERNEL_FILL, s, [&] { return launch_fill(f, s); });
    if (e != hipSuccess) return hip_fail(e, "fill launch");
  }
  return SRA_OK;
}

sra_status set_error(sra_status s, const char* msg) { return fail(s, msg); }

}  // namespace sra

extern "C" {

sra_status sra_forward(const sra_problem* p, const void* q_gen, const void* k_gen, const void* v_gen,
                       const void* q_ref, const void* k_ref, const void* v_ref, void* o_gen, void* o_ref,
                       float* lse_gen, float* lse_ref, void* workspace, size_t workspace_bytes,
                       void* stream) {
  return sra::forward_call(p, q_gen, k_gen, v_gen, q_ref, k_ref, v_ref, o_gen, o_ref, lse_gen, lse_ref,
                           workspace, workspace_bytes, stream, nullptr, 0);
}

sra_status sra_backward(const sra_problem* p, const void* q_gen, const void* k_gen, const void* v_gen,
                        const void* q_ref, const void* k_ref, const void* v_ref, const void* o_gen,
                        const void* o_ref, const float* lse_gen, const float* lse_ref, const void* do_gen,
                        const void* do_ref, void* dq_gen, void* dk_gen, void* dv_gen, void* dq_ref,
                        void* dk_ref, void* dv_ref, void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  Layout L;
  std::shared_ptr<CachedPlan> cp;
  sra_status st = common_checks(p, &L, &cp);
  if (st != SRA_OK) return st;
  st = L.gen_only ? check_tensors(L, {q_gen, k_gen, v_gen, o_gen, lse_gen, do_gen, dq_gen, dk_gen, dv_gen},
                                  {k_ref, v_ref, dk_ref, dv_ref})
                  : check_tensors(L, {q_gen, k_gen, v_gen, o_gen, lse_gen, do_gen, dq_gen, dk_gen, dv_gen},
                                  {q_ref, k_ref, v_ref, o_ref, lse_ref, do_ref, dq_ref, dk_ref, dv_ref});
  if (st != SRA_OK) return st;
  const size_t need = bwd_workspace(*cp);
  if (workspace_bytes < need)
    return fail(SRA_ERR_WORKSPACE_TOO_SMALL, "backward needs " + std::to_string(need) + " workspace bytes");
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) % kAlign))
    return fail(SRA_ERR_INVALID_ARGUMENT, "workspace must be non-NULL and 256-byte aligned");

  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  st = cache().upload(cp->bwd, ws, s);
  if (st != SRA_OK) return st;
  hipError_t e;
  const Plan& P = cp->plan;
  const Layout& E = P.exec;
  const int32_t row_elems = L.heads * L.head_dim;
  const size_t gen_stat = stat_bytes(E, E.sum_gen);
  const size_t ref_stat = stat_bytes(E, E.sum_ref);
  float* ndelta_gen = reinterpret_cast<float*>(ws + cp->bwd.bytes);
  float* lse2_gen = reinterpret_cast<float*>(ws + cp->bwd.bytes + gen_stat);
  float* ndelta_ref = reinterpret_cast<float*>(ws + cp->bwd.bytes + 2 * gen_stat);
  float* lse2_ref = reinterpret_cast<float*>(ws + cp->bwd.bytes + 2 * gen_stat + ref_stat);

  // the reference tensors the kernels use: the caller's, or their compacted copies
  const __bf16* ref_in[5] = {static_cast<const __bf16*>(q_ref), static_cast<const __bf16*>(k_ref),
                             static_cast<const __bf16*>(v_ref), static_cast<const __bf16*>(o_ref),
                             static_cast<const __bf16*>(do_ref)};
  __bf16* ref_out[3] = {static_cast<__bf16*>(dq_ref), static_cast<__bf16*>(dk_ref), static_cast<__bf16*>(dv_ref)};
  const float* ref_lse = lse_ref;
  int64_t ref_stride = L.ref_stride;
  if (P.compacted) {
    char* c = ws + cp->bwd.bytes + 2 * gen_stat + 2 * ref_stat;
    const size_t rb = rows_bytes(E, E.sum_ref);
    GatherArgs g{};
    g.index = reinterpret_cast<const int32_t*>(ws + cp->bwd.offsets[5]);
    g.rows = int32_t(E.sum_ref);
    g.row_elems = row_elems;
    g.heads = L.heads;
    for (int t = 0; t < 5; ++t) {
      // q, o and do of the reference rows are not read when reference tokens are not queries
      const bool used = !(L.gen_only && (t == 0 || t == 3 || t == 4));
      g.src[t] = used ? ref_in[t] : nullptr;
      g.src_stride[t] = t < 3 ? L.ref_stride : row_elems;
      g.dst[t] = reinterpret_cast<__bf16*>(c + t * rb);
      ref_in[t] = used ? g.dst[t] : nullptr;
    }
    float* lse_c = reinterpret_cast<float*>(c + 8 * rb);
    if (!L.gen_only) {
      g.lse_src = lse_ref;
      g.lse_src_rows = int32_t(L.sum_ref);
      g.lse_dst = lse_c;
    }
    e = timed(SRA_KERNEL_GATHER, s, [&] { return launch_gather(g, s); });
    if (e != hipSuccess) return hip_fail(e, "gather launch");
    for (int t = 0; t < 3; ++t) ref_out[t] = reinterpret_cast<__bf16*>(c + (5 + t) * rb);
    ref_lse = L.gen_only ? nullptr : lse_c;
    ref_stride = row_elems;
  }

  DeltaArgs d{};
  d.o[0] = static_cast<const __bf16*>(o_gen);
  d.o[1] = ref_in[3];
  d.dout[0] = static_cast<const __bf16*>(do_gen);
  d.dout[1] = ref_in[4];
  d.lse[0] = lse_gen;
  d.lse[1] = ref_lse;
  d.ndelta[0] = ndelta_gen;
  d.ndelta[1] = ndelta_ref;
  d.lse2[0] = lse2_gen;
  d.lse2[1] = lse2_ref;
  d.rows[0] = int32_t(E.sum_gen);
  d.rows[1] = L.gen_only ? 0 : int32_t(E.sum_ref);  // no ref query rows when gen-only
  d.heads = L.heads;
  e = timed(SRA_KERNEL_DELTA, s, [&] { return launch_delta(d, L.head_dim, s); });
  if (e != hipSuccess) return hip_fail(e, "delta launch");

  BwdArgs a{};
  a.q[0] = static_cast<const __bf16*>(q_gen);
  a.k[0] = static_cast<const __bf16*>(k_gen);
  a.v[0] = static_cast<const __bf16*>(v_gen);
  a.q[1] = ref_in[0];
  a.k[1] = ref_in[1];
  a.v[1] = ref_in[2];
  a.in_stride[0] = L.gen_stride;
  a.in_stride[1] = ref_stride;
  a.dout[0] = static_cast<const __bf16*>(do_gen);
  a.dout[1] = ref_in[4];
  a.lse2[0] = lse2_gen;
  a.lse2[1] = lse2_ref;
  a.ndelta[0] = ndelta_gen;
  a.ndelta[1] = ndelta_ref;
  a.dq[0] = static_cast<__bf16*>(dq_gen);
  a.dk[0] = static_cast<__bf16*>(dk_gen);
  a.dv[0] = static_cast<__bf16*>(dv_gen);
  a.dq[1] = ref_out[0];
  a.dk[1] = ref_out[1];
  a.dv[1] = ref_out[2];
  a.rows[0] = int32_t(E.sum_gen);
  a.rows[1] = int32_t(E.sum_ref);
  a.heads = L.heads;
  a.scale = L.scale;
  a.scale_log2 = float(double(L.scale) * 1.4426950408889634);

  a.items = reinterpret_cast<const WorkItem*>(ws + cp->bwd.offsets[2]);
  a.spans = reinterpret_cast<const Span*>(ws + cp->bwd.offsets[3]);
  e = timed(SRA_KERNEL_DKDV, s, [&] { return launch_dkv(a, int(P.dkv.items.size()), L.head_dim, s); });
  if (e != hipSuccess) return hip_fail(e, "dkv launch");
  a.items = reinterpret_cast<const WorkItem*>(ws + cp->bwd.offsets[0]);
  a.spans = reinterpret_cast<const Span*>(ws + cp->bwd.offsets[1]);
  e = timed(SRA_KERNEL_DQ, s, [&] { return launch_dq(a, int(P.dq.items.size()), L.head_dim, s); });
  if (e != hipSuccess) return hip_fail(e, "dq launch");
  if (!P.fill.empty()) {
    FillArgs f{};
    f.ranges = reinterpret_cast<const FillRange*>(ws + cp->bwd.offsets[4]);
    f.n_ranges = int32_t(P.fill.size());
    f.heads = L.heads;
    f.head_dim = L.head_dim;
    f.t[0] = L.gen_only ? nullptr : ref_out[0];
    f.t[1] = ref_out[1];
    f.t[2] = ref_out[2];
    e = timed(SRA_KERNEL_FILL, s, [&] { return launch_fill(f, s); });
    if (e != hipSuccess) return hip_fail(e, "fill launch");
  }
  if (P.compacted) {
    ScatterArgs sc{};
    sc.index = reinterpret_cast<const int32_t*>(ws + cp->bwd.offsets[6]);
    sc.rows = int32_t(L.sum_ref);
    sc.row_elems = row_elems;
    sc.heads = L.heads;
    for (int t = 0; t < 3; ++t) sc.src[t] = ref_out[t];
    sc.dst[0] = L.gen_only ? nullptr : static_cast<__bf16*>(dq_ref);
    sc.dst[1] = static_cast<__bf16*>(dk_ref);
    sc.dst[2] = static_cast<__bf16*>(dv_ref);
    e = timed(SRA_KERNEL_SCATTER, s, [&] { return launch_scatter(sc, s); });
    if (e != hipSuccess) return hip_fail(e, "scatter launch");
  }
  return SRA_OK;
}

sra_status sra_pair_counts(const sra_problem* p, int64_t* gen_pairs, int64_t* ref_pairs) {
  g_last_error.clear();
  Layout L;
  std::string err;
  sra_status st = make_layout(p, &L, &err);
  if (st != SRA_OK) return fail(st, err);
  closed_form_pairs(L, gen_pairs, ref_pairs);
  return SRA_OK;
}

sra_status sra_dense_mask(const sra_problem* p, int32_t sample, uint8_t* out) {
  g_last_error.clear();
  Layout L;
  std::string err;
  sra_status st = make_layout(p, &L, &err);
  if (st != SRA_OK) return fail(st, err);
  if (sample < 0 || sample >= L.batch) return fail(SRA_ERR_INVALID_ARGUMENT, "sample out of range");
  if (!out) return fail(SRA_ERR_INVALID_ARGUMENT, "out is NULL");
  const SampleLayout& sm = L.samples[sample];
  const int64_t G = sm.G, R = sm.R, n = G + R;
  std::vector<uint8_t> valid(size_t(R), 0);  // reference token takes part (its frame and its own entry)
  for (const auto& r : sm.vruns)
    for (int64_t j = r.first; j < r.second; ++j) valid[size_t(j)] = 1;
  const int64_t gsz = sm.F * sm.group;  // reference tokens per self-attention group
  for (int64_t q = 0; q < n; ++q) {
    uint8_t* row = out + q * n;
    if (q < G) {  // generation query: gen keys (within the window, if any), every valid ref key
      for (int64_t k = 0; k < G; ++k)
        row[k] = sm.window < 0 || std::llabs(q / sm.Fg - k / sm.Fg) <= sm.window;
      for (int64_t j = 0; j < R; ++j) row[G + j] = valid[size_t(j)];
    } else {  // reference query: no gen key; the valid ref keys of its own group if it is valid
      const int64_t i = q - G;
      std::memset(row, 0, size_t(n));
      if (!valid[size_t(i)]) continue;
      const int64_t g0 = i / gsz * gsz, g1 = std::min(R, g0 + gsz);
      for (int64_t j = g0; j < g1; ++j) row[G + j] = valid[size_t(j)];
    }
  }
  return SRA_OK;
}

static const Schedule* pick(const Plan& P, int which) {
  switch (which) {
    case SRA_SCHED_FORWARD: return &P.fwd;
    case SRA_SCHED_BWD_DQ: return &P.dq;
    case SRA_SCHED_BWD_DKDV: return &P.dkv;
    default: return nullptr;
  }
}

sra_status sra_schedule_info(const sra_problem* p, int which, int64_t* n_items, int64_t* n_spans,
                             int64_t* covered) {
  g_last_error.clear();
  Layout L;
  std::string err;
  sra_status st = make_layout(p, &L, &err);
  if (st != SRA_OK) return fail(st, err);
  Plan P;
  build_plan(L, &P);
  const Schedule* S = pick(P, which);
  if (!S) return fail(SRA_ERR_INVALID_ARGUMENT, "unknown schedule");
  if (n_items) *n_items = int64_t(S->items.size());
  if (n_spans) *n_spans = int64_t(S->spans.size());
  if (covered) *covered = covered_pairs(*S, which == SRA_SCHED_BWD_DKDV);
  return SRA_OK;
}

sra_status sra_schedule_mask(const sra_problem* p, int which, int32_t sample, uint8_t* out) {
  g_last_error.clear();
  Layout L;
  std::string err;
  sra_status st = make_layout(p, &L, &err);
  if (st != SRA_OK) return fail(st, err);
  if (sample < 0 || sample >= L.batch) return fail(SRA_ERR_INVALID_ARGUMENT, "sample out of range");
  if (!out) return fail(SRA_ERR_INVALID_ARGUMENT, "out is NULL");
  Plan P;
  build_plan(L, &P);
  const Schedule* S = pick(P, which);
  if (!S) return fail(SRA_ERR_INVALID_ARGUMENT, "unknown schedule");
  const SampleLayout& sm = L.samples[sample];
  const int64_t n = sm.G + sm.R;
  std::memset(out, 0, size_t(n * n));
  auto local = [&](int32_t stream, int64_t row) -> int64_t {  // packed row -> [gen ; ref] index
    if (stream == 0) return row - sm.gen_off;
    if (P.compacted) {  // a row of the compacted reference stream: map it back
      if (row < 0 || row >= int64_t(P.ref_gather.size())) return -1;
      row = P.ref_gather[size_t(row)];
    }
    return sm.G + (row - sm.ref_off);
  };
  const bool key_major = which == SRA_SCHED_BWD_DKDV;
  for (const WorkItem& w : S->items) {
    if (w.stream < 0 || w.head != 0 || w.sample != sample) continue;
    for (int32_t si = 0; si < w.span_cnt; ++si) {
      const Span& sp = S->spans[w.span_off + si];
      // a key-major span may reach only the item's keys [lo, hi)
      const int32_t a0 = sp.keys ? (sp.keys & 0xffff) : 0, a1 = sp.keys ? (sp.keys >> 16) : w.len;
      if (a0 < 0 || a1 > w.len || a0 >= a1) return fail(SRA_ERR_INTERNAL, "span key range outside its item");
      for (int32_t a = a0; a < a1; ++a) {
        const int64_t ta = local(w.stream, int64_t(w.start) + a);
        for (int32_t b = 0; b < sp.len; ++b) {
          const int64_t tb = local(sp.stream, int64_t(sp.start) + b);
          if (ta < 0 || ta >= n || tb < 0 || tb >= n) return fail(SRA_ERR_INTERNAL, "schedule leaves its sample");
          const int64_t q = key_major ? tb : ta, k = key_major ? ta : tb;
          uint8_t& c = out[q * n + k];
          if (c < 255) ++c;
        }
      }
    }
  }
  return SRA_OK;
}

sra_status sra_schedule_export(const sra_problem* p, int which, int32_t* items, int64_t items_capacity,
                               int32_t* spans, int64_t spans_capacity) {
  g_last_error.clear();
  Layout L;
  std::string err;
  sra_status st = make_layout(p, &L, &err);
  if (st != SRA_OK) return fail(st, err);
  Plan P;
  build_plan(L, &P);
  const Schedule* S = pick(P, which);
  if (!S) return fail(SRA_ERR_INVALID_ARGUMENT, "unknown schedule");
  if (items) {
    if (items_capacity < int64_t(S->items.size()) * 8) return fail(SRA_ERR_INVALID_ARGUMENT, "items buffer too small");
    std::memcpy(items, S->items.data(), S->items.size() * sizeof(WorkItem));
  }
  if (spans) {
    if (spans_capacity < int64_t(S->spans.size()) * 4) return fail(SRA_ERR_INVALID_ARGUMENT, "spans buffer too small");
    std::memcpy(spans, S->spans.data(), S->spans.size() * sizeof(Span));
  }
  return SRA_OK;
}

sra_status sra_kernel_timing_enable(int enable) {
  g_last_error.clear();
  timer().enable(enable != 0);
  return SRA_OK;
}

sra_status sra_kernel_timing(int kernel, double* total_ms, int64_t* launches) {
  g_last_error.clear();
  if (kernel < 0 || kernel >= SRA_KERNEL_COUNT) return fail(SRA_ERR_INVALID_ARGUMENT, "unknown kernel id");
  timer().read(kernel, total_ms, launches);
  return SRA_OK;
}

sra_status sra_release_caches(void) {
  g_last_error.clear();
  cache().clear();
  resident().clear();
  return SRA_OK;
}

const char* sra_status_string(sra_status s) {
  switch (s) {
    case SRA_OK: return "SRA_OK";
    case SRA_ERR_INVALID_ARGUMENT: return "SRA_ERR_INVALID_ARGUMENT";
    case SRA_ERR_UNSUPPORTED: return "SRA_ERR_UNSUPPORTED";
    case SRA_ERR_WORKSPACE_TOO_SMALL: return "SRA_ERR_WORKSPACE_TOO_SMALL";
    case SRA_ERR_HIP: return "SRA_ERR_HIP";
    case SRA_ERR_INTERNAL: return "SRA_ERR_INTERNAL";
  }
  return "SRA_ERR_UNKNOWN";
}

const char* sra_last_error(void) { return g_last_error.c_str(); }

int32_t sra_version(void) { return 200; }

}  // extern "C"
