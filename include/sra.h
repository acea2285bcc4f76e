/*
 * sra.h — C ABI of libsra: Sparse Reference Attention (SRA) on AMD Instinct MI355X (gfx950).
 *
 * SRA is the asymmetric attention of Avatar V (§1 contributions; §2.1 "Sparse Reference
 * Attention"; §4.3 reference KV caching and invalid-token skipping; §8 related work):
 *   - every generation (gen) query attends to all gen keys of its sample and to every valid
 *     reference (ref) key of its sample, through ONE softmax over the concatenated key set
 *     (§4.3 concatenates the cached reference K/V with the generation K/V);
 *   - every ref query attends only to the ref keys of its own self-attention group, never to
 *     gen keys (§1, §8.2: the reference side attends only within itself). A group is `group_frames`
 *     consecutive reference latent frames; group_frames = 1 keeps the cost linear in the
 *     reference length (§1, §2.1);
 *   - tokens of invalid reference frames (§4.3, e.g. frames where the face is not visible),
 *     and single reference tokens marked invalid, are neither keys nor queries: their
 *     outputs are 0, their log-sum-exp is -inf and their gradients are 0.
 * Samples of a packed (varlen) batch never see each other.
 *
 * Conventions shared by every entry point
 *   Tensors   bf16 tensors are [tokens, heads, head_dim] with head stride head_dim and element
 *             stride 1. Tokens of all samples are packed back to back in sample order, and
 *             frame-major (frame, row, column) inside a sample. q/k/v of a stream use that
 *             stream's token stride (elements between consecutive tokens, >= heads*head_dim,
 *             so q/k/v packed into one buffer work); o, do, dq, dk, dv are dense
 *             (token stride heads*head_dim). lse tensors are fp32 [heads, tokens], natural log.
 *   Memory    every data pointer and the workspace are DEVICE pointers owned by the caller.
 *             The library allocates no device memory. It owns pinned host staging buffers for
 *             its cached schedules (reused across plans, freed by sra_release_caches or at
 *             process exit); a geometry not seen before costs one host planning pass and, when
 *             no staging buffer is free, one hipHostMalloc (the cache holds 256 plans).
 *   Streams   `stream` is a hipStream_t (NULL = the default stream). Calls only enqueue work
 *             on it and never synchronise the device.
 *   Errors    every argument is validated before anything is enqueued, so a call that
 *             returns an error has written nothing. sra_last_error() gives a per-thread
 *             message. No C++ exception crosses this boundary. All functions are thread safe.
 *   Supported head_dim in {64, 128}; heads >= 1; batch >= 1; every sample has >= 1 gen token.
 *   Limits    packed tokens of each stream <= 2^31 - 1 (beyond: SRA_ERR_INVALID_ARGUMENT);
 *             num_heads * packed tokens of each stream <= 2^31 - 1 (beyond: SRA_ERR_UNSUPPORTED;
 *             per-row statistics are indexed in 32 bits); token strides <= (2^31 - 1) / 64
 *             elements (beyond: SRA_ERR_UNSUPPORTED; offsets inside a tile are 32-bit). Tensors
 *             themselves may exceed 2^31 elements: token offsets are 64-bit.
 */
#ifndef SRA_H_
#define SRA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum sra_status {
  SRA_OK = 0,
  SRA_ERR_INVALID_ARGUMENT = 1,     /* bad geometry, null pointer, stride, flag, ...           */
  SRA_ERR_UNSUPPORTED = 2,          /* valid request the library does not implement (head_dim) */
  SRA_ERR_WORKSPACE_TOO_SMALL = 3,  /* workspace_bytes below sra_workspace_size()              */
  SRA_ERR_HIP = 4,                  /* the HIP runtime reported an error while enqueuing       */
  SRA_ERR_INTERNAL = 5              /* host allocation failure or internal inconsistency       */
} sra_status;

/* Geometry of one sample (host memory). Gen tokens G = gen_frames*gen_h*gen_w (>= 1);
 * ref tokens R = ref_frames*ref_h*ref_w (>= 0); F = ref_h*ref_w tokens per ref frame. */
typedef struct sra_sample_geom {
  int32_t gen_frames, gen_h, gen_w;
  int32_t ref_frames, ref_h, ref_w;
  int32_t group_frames;              /* >= 1: ref frames per ref self-attention group          */
  int32_t gen_window;                /* with SRA_FLAG_GEN_WINDOW: >= 0, see below; else ignored */
  const uint8_t* ref_frame_valid;    /* host, ref_frames bytes (0 = invalid); NULL = all valid */
  const uint8_t* ref_token_valid;    /* host, R bytes, frame-major (0 = invalid token); NULL =
                                        every token of a valid frame. A ref token takes part iff
                                        its frame and its own entry are valid (§4.3 invalid
                                        tokens); invalid tokens are treated like tokens of
                                        invalid frames. */
} sra_sample_geom;

typedef struct sra_problem {
  int32_t batch;                     /* samples in the packed batch, >= 1                      */
  int32_t num_heads;                 /* H >= 1 (same for Q, K and V)                           */
  int32_t head_dim;                  /* d in {64, 128}                                         */
  float softmax_scale;               /* <= 0 selects 1/sqrt(head_dim)                          */
  const sra_sample_geom* samples;    /* host array [batch]                                     */
  int64_t gen_token_stride;          /* elements between gen q/k/v tokens; 0 selects H*d       */
  int64_t ref_token_stride;          /* elements between ref q/k/v tokens; 0 selects H*d       */
  uint32_t flags;                    /* 0 or SRA_FLAG_* bits                                   */
} sra_problem;

/* Problem flags.
 * SRA_FLAG_GEN_QUERIES_ONLY: reference tokens are context only, not queries. This is the
 *   inference path of cached reference K/V (§4.3): across denoising steps the reference
 *   tokens' own outputs do not change, so only the generation rows are computed. The
 *   forward writes o_gen and lse_gen only; q_ref, o_ref and lse_ref are not read or written
 *   and may be NULL. The backward is that of the gen rows alone (equivalently: do_ref = 0):
 *   it writes dq_gen, dk_gen, dv_gen, dk_ref and dv_ref; q_ref, o_ref, lse_ref, do_ref and
 *   dq_ref are not touched and may be NULL. Pair counts and schedules omit the ref queries.
 * SRA_FLAG_GEN_WINDOW: temporal window on generation-to-generation attention, the sparse
 *   temporal attention of the super-resolution refiner (§2.4, which restricts each frame's
 *   receptive field to a local neighbourhood of frames and gives no width): a gen query in
 *   gen latent frame t sees the gen keys of frames t' with |t - t'| <= gen_window of its
 *   sample, and still every valid reference key. Reference queries are unchanged. */
enum { SRA_FLAG_GEN_QUERIES_ONLY = 1u, SRA_FLAG_GEN_WINDOW = 2u };

/* Which schedule an inspection hook looks at. */
enum {
  SRA_SCHED_FORWARD = 0,   /* query tiles -> key spans (forward pass)                 */
  SRA_SCHED_BWD_DQ = 1,    /* query tiles -> key spans (dQ kernel of the backward)    */
  SRA_SCHED_BWD_DKDV = 2   /* key tiles -> query spans (dK/dV kernel of the backward) */
};

/* Bytes of device workspace sra_forward (backward = 0) or sra_backward (backward = 1) needs
 * for problem `p`. Writes *bytes; host only, enqueues nothing. */
sra_status sra_workspace_size(const sra_problem* p, int backward, size_t* bytes);

/* Forward pass of SRA (the definition at the top of this file).
 * In : q_gen, k_gen, v_gen  bf16 [sumG, H, d] (gen token stride);
 *      q_ref, k_ref, v_ref  bf16 [sumR, H, d] (ref token stride); may be NULL when sumR = 0.
 * Out: o_gen bf16 [sumG, H, d], o_ref bf16 [sumR, H, d] (dense);
 *      lse_gen fp32 [H, sumG], lse_ref fp32 [H, sumR]: natural-log log-sum-exp of the scaled
 *      logits of each query row (-inf for rows of invalid frames).
 * workspace: device buffer of at least sra_workspace_size(p, 0) bytes, 256-byte aligned; its
 * contents are scratch and need no initialisation. Every output element is written. */
sra_status sra_forward(const sra_problem* p,
                       const void* q_gen, const void* k_gen, const void* v_gen,
                       const void* q_ref, const void* k_ref, const void* v_ref,
                       void* o_gen, void* o_ref, float* lse_gen, float* lse_ref,
                       void* workspace, size_t workspace_bytes, void* stream);

/* Backward pass (§3.3: personality SFT trains the model with Sparse Reference Attention in the
 * loop, so the method needs the gradient of the attention of the top of this file; it is the
 * gradient of masked softmax attention, which the paper does not spell out).
 * Gradients of the forward outputs o_gen/o_ref with respect to every input,
 * given the upstream gradients do_gen/do_ref (bf16, dense, same shapes as o) and the forward's
 * o and lse (as sra_forward wrote them). Writes dq/dk/dv for both streams (bf16, dense,
 * same shapes as q/k/v); it overwrites them and does not accumulate. Gradients of tokens of
 * invalid frames are 0. Internally: D = rowsum(dO * O) in fp32, then the dK/dV and dQ
 * products of the softmax gradient with fp32 accumulation.
 * workspace: at least sra_workspace_size(p, 1) bytes, 256-byte aligned, no initialisation. */
sra_status sra_backward(const sra_problem* p,
                        const void* q_gen, const void* k_gen, const void* v_gen,
                        const void* q_ref, const void* k_ref, const void* v_ref,
                        const void* o_gen, const void* o_ref,
                        const float* lse_gen, const float* lse_ref,
                        const void* do_gen, const void* do_ref,
                        void* dq_gen, void* dk_gen, void* dv_gen,
                        void* dq_ref, void* dk_ref, void* dv_ref,
                        void* workspace, size_t workspace_bytes, void* stream);

/* ---- allocation-free forward ------------------------------------------------------------ */

/* Size in bytes of the library's static device scratch array, the workspace of
 * sra_forward_noalloc (one array per device, held from the first such call on that device until
 * the process ends). */
#define SRA_NOALLOC_WORKSPACE_MAX (32u << 20)

/* For callers that cannot allocate device memory (code under stream capture, tight serving
 * loops, harnesses that forbid hipMalloc): sra_forward with the workspace taken from the
 * library's static scratch array on the current device instead of a caller buffer. Same
 * kernels, so results are bitwise those of sra_forward.
 * In/out tensors, stream and validation as sra_forward; `stream` must belong to the current
 * device (else SRA_ERR_INVALID_ARGUMENT). A problem whose workspace (sra_workspace_size with
 * backward = 0) exceeds SRA_NOALLOC_WORKSPACE_MAX is rejected with SRA_ERR_WORKSPACE_TOO_SMALL
 * before anything is enqueued: in practice every problem whose token masks do not force the
 * compacted reference stream fits (the 720p layer needs 0.8 MB).
 * Allocates no device memory and no pinned host memory (no hipMalloc, hipHostMalloc or
 * hipFree): the schedule tables are copied from the plan's host image, and not at all when the
 * previous sra_forward_noalloc call on this device used the same geometry and stream (the
 * array keeps the last call's tables). A geometry not seen before is planned in host heap
 * memory, as for every entry point.
 * All calls on one device share one array: calls that overlap on a device (different streams
 * or threads without ordering between them) race and may read each other's tables. The first
 * call on a device loads the array there (a one-time cost of milliseconds). */
sra_status sra_forward_noalloc(const sra_problem* p,
                               const void* q_gen, const void* k_gen, const void* v_gen,
                               const void* q_ref, const void* k_ref, const void* v_ref,
                               void* o_gen, void* o_ref, float* lse_gen, float* lse_ref,
                               void* stream);

/* ---- host-only inspection hooks (no device needed; used to test the schedules) ---------- */

/* Visible (query, key) pairs per head summed over samples: the work of the attention, which
 * §1 and §2.1 state grows (almost) linearly with the reference length; from the closed form
 * G*(G + R_valid) for gen queries (G*R_valid plus the window's gen pairs with
 * SRA_FLAG_GEN_WINDOW) and sum over groups of (valid tokens of the group)^2 for ref queries.
 * Either output pointer may be NULL. */
sra_status sra_pair_counts(const sra_problem* p, int64_t* gen_pairs, int64_t* ref_pairs);

/* The visibility rule of the top of this file (§1, §2.1, §4.3; the window of §2.4 with
 * SRA_FLAG_GEN_WINDOW) written out for `sample` as a (G+R) x (G+R) byte matrix, rows = queries
 * and columns = keys in [gen ; ref] order of that sample: out[q*(G+R)+k] = 1 when query q sees
 * key k, else 0. Computed from the geometry alone (not from a schedule; sra_schedule_mask
 * gives what a schedule covers). Other flags do not change it. out must hold (G+R)^2 bytes
 * (host memory owned by the caller); host only. */
sra_status sra_dense_mask(const sra_problem* p, int32_t sample, uint8_t* out);

/* Sizes of schedule `which` (SRA_SCHED_*), the tile schedules that realise the visibility rule
 * of §1, §2.1 and §4.3 without a dense mask: work items (all heads) and span entries, and the
 * (query, key) pairs the schedule covers per head (must equal the pair count). */
sra_status sra_schedule_info(const sra_problem* p, int which, int64_t* n_items,
                             int64_t* n_spans, int64_t* covered_pairs);

/* Expands schedule `which` (the visibility rule of §1, §2.1 and §4.3 as tiles) for head 0 of
 * `sample` into a (G+R) x (G+R) byte matrix, rows =
 * queries and columns = keys in [gen ; ref] order of that sample: out[q*(G+R)+k] = number of
 * work items that compute the pair (q, k), so a correct schedule gives exactly the 0/1
 * visibility mask. out must hold (G+R)^2 bytes (host). */
sra_status sra_schedule_mask(const sra_problem* p, int which, int32_t sample, uint8_t* out);

/* Copies schedule `which` (the tiles realising §1, §2.1 and §4.3) into host buffers:
 * items[8*i + 0..7] = {stream, head, start, length,
 * span_offset, span_count, sample, reserved} per work item, spans[4*j + 0..3] = {stream,
 * start, length, keys} per span (stream 0 = gen, 1 = ref; start = packed token row; keys, in
 * the dK/dV schedule only: the item's keys [lo, hi), counted from its first key, that the
 * span's queries see, packed lo | hi << 16, or 0 for all of them).
 * items/spans may be NULL to query only; capacities count int32 elements.
 * Items are listed in launch order (item i runs on XCD i % 8). When the head count is a
 * multiple of 8, an item whose first span is its sample's gen rows may start that span part
 * way in and wrap around (the span then appears as two entries, its tail first), so that the
 * items resident on one XCD stream the same rows at the same time; the rows covered are the
 * same either way.
 * When token masks split reference frames into more runs of valid tokens than there are
 * groups with a valid token, the library runs on the compacted reference stream (the valid
 * reference tokens of the batch back to back, in sample, group and token order: gathered
 * before the kernels, outputs scattered back after); ref rows of the schedule are then rows
 * of that stream. */
sra_status sra_schedule_export(const sra_problem* p, int which, int32_t* items,
                               int64_t items_capacity, int32_t* spans, int64_t spans_capacity);

/* ---- per-kernel timing (tracing hook; library infrastructure, no passage of the paper) --- */

/* Kernels of the library, for sra_kernel_timing. */
enum {
  SRA_KERNEL_FORWARD = 0,   /* forward pass                              */
  SRA_KERNEL_DELTA = 1,     /* backward: D = rowsum(dO * O)              */
  SRA_KERNEL_DKDV = 2,      /* backward: dK and dV (key-major)           */
  SRA_KERNEL_DQ = 3,        /* backward: dQ (query-major)                */
  SRA_KERNEL_FILL = 4,      /* rows of invalid reference frames          */
  SRA_KERNEL_GATHER = 5,    /* reference rows into the compacted stream  */
  SRA_KERNEL_SCATTER = 6,   /* compacted rows back to the reference rows */
  SRA_KERNEL_COUNT = 7
};

/* enable != 0: from now on every kernel launch is bracketed by two hipEvents recorded on the
 * caller's stream, and the accumulated totals are reset. enable == 0 stops recording. */
sra_status sra_kernel_timing_enable(int enable);

/* Waits for the recorded events and returns the summed duration (ms) and launch count of
 * kernel `kernel` (SRA_KERNEL_*) since timing was enabled. */
sra_status sra_kernel_timing(int kernel, double* total_ms, int64_t* launches);

/* Library infrastructure (no passage of the paper). Frees cached schedules and their pinned
 * host staging buffers, after waiting for the copies that read them (the only entry point that
 * waits on the device). Evicting a plan from the cache neither waits nor frees: its staging
 * buffer is reused for a later plan once the copies out of it have completed. Safe to call at
 * any time; later calls rebuild what they need. */
sra_status sra_release_caches(void);

/* Library infrastructure (no passage of the paper): status names, the per-thread detail of
 * the last failing call ("" if none), and the version as major*10000 + minor*100 + patch. */
const char* sra_status_string(sra_status s);
const char* sra_last_error(void);
int32_t sra_version(void);

#ifdef __cplusplus
}
#endif
#endif /* SRA_H_ */
