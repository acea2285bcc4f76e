// Library-internal entry points shared by the C ABI translation units.
#pragma once
#include <stddef.h>

#include "sra.h"

namespace sra {

// The device workspace of the allocation-free forward: the library's static scratch array on
// the current device (its address as hipGetSymbolAddress gave it) and its size.
struct StaticWorkspace {
  void* ptr;
  size_t bytes;
  int device;
};

// Fills the static workspace of the stream's device (called only after the problem passed
// validation and fits in `bytes`); returns SRA_OK or an error with the message set.
typedef sra_status (*StaticWorkspaceFn)(void* stream, StaticWorkspace* sw);

// sra_forward, or with `static_ws` (not null) the allocation-free forward: problems needing
// more than `static_bytes` are rejected before any device call, the caller's workspace
// arguments are ignored, the workspace is the one static_ws gives, and the schedule is copied
// from pageable host memory only when it is not already resident there.
sra_status forward_call(const sra_problem* p, const void* q_gen, const void* k_gen, const void* v_gen,
                        const void* q_ref, const void* k_ref, const void* v_ref, void* o_gen, void* o_ref,
                        float* lse_gen, float* lse_ref, void* workspace, size_t workspace_bytes, void* stream,
                        StaticWorkspaceFn static_ws, size_t static_bytes);

// Sets the thread's last-error message and returns `s`.
sra_status set_error(sra_status s, const char* msg);

}  // namespace sra
