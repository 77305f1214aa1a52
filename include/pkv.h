/*
 * pkv.h -- C ABI of libpkv: the fused suffix restore of PatchKV on MI355X.
 *
 * After a middle edit C_old = P + M_old + S  ->  C_new = P + M_new + S
 * (PatchKV, Eq. 1), the blocks of the aligned suffix S that are not in the
 * repair set R (Eq. 12) are restored from a quantized checkpoint: each block
 * is decoded by its frozen precision tag (Eq. 14), its keys are re-phased by
 * the edit shift Delta (Eq. 3; values are never rotated), and its rows are
 * written into the request's destination KV pages (Section IV-D, the fused
 * dequantize-and-scatter of the resume path, Section IV-A step 5).
 *
 * Usage: build an immutable plan once per resume (host validation, tile
 * list, device metadata), launch it on a HIP stream as often as wanted, free
 * it.  Every pointer in this header is a plain host or device address; no
 * framework types appear.
 *
 * ----------------------------------------------------------------------------
 * Checkpoint format (one request; all sizes follow from pkv_model_t and the
 * request's tags -- pkv_payload_size() computes them):
 *
 *  payload (device, bytes): for each layer l = 0..L-1, for each tag in the
 *    order FP16, K8V8, K8V4, K4V4, for each block b with that tag in
 *    ascending order (repair blocks included; their bytes are never read):
 *    the block's K tile, then its V tile.  A tile is the block's B rows in
 *    token-major order [B][H][D] (rows past the end of the suffix in the last
 *    block are padding).  Channel formats: FP16 = IEEE binary16; 8-bit = one
 *    unsigned code per channel; 4-bit = two codes per byte, channel 2j in the
 *    low nibble of byte j.  Same-tag blocks therefore form one contiguous run
 *    per layer (the clustered runs of Section IV-D).
 *
 *  scales (device, binary16): [L][NB][H][2 (K, V)][2 (scale, zero)].  A
 *    quantized channel decodes as code * scale + zero.  Entries of FP16
 *    blocks are ignored.
 *
 *  caches (device), of the output dtype (binary16 or bfloat16), in one of two
 *    layouts (pkv_model_t.kv_layout):
 *      PKV_KV_SEPARATE: k_cache and v_cache, each [L][pool_pages][P][H][D];
 *      PKV_KV_PAIRED:   one allocation [L][pool_pages][2][P][H][D], the K
 *        slots of a page followed by its V slots; k_cache is its start and
 *        v_cache = k_cache + P*H*D elements.
 *    Token t of block b of a request lands on logical row r = dst_row0 +
 *    b*B + t, slot r % P of physical page page_table[r / P].  Nothing else
 *    is written: rows of repair blocks, padding rows, prefix rows and pages
 *    owned by nobody keep their bytes.
 *
 * Arithmetic: decode exact; keys rotated in double precision with a
 * double-precision cos/sin(Delta * f_i) table over the model's rotary pairs
 * and frequencies f_i (pkv_rope_style_t, rotary_dim and inv_freq in
 * pkv_model_t); values decoded in single precision; one round-to-nearest-even
 * to the output dtype after an intermediate single-precision value.  So every
 * element is the exactly rounded result, except within the double-rounding
 * window of a rounding midpoint (about 2^-24 relative), where it may be the
 * midpoint's other neighbour.  When Delta == 0 keys are not rotated at all
 * (R(0) = I), so the FP16 tag with Delta == 0 and fp16 output is a bit-exact
 * copy.
 * ----------------------------------------------------------------------------
 */
#ifndef PKV_H
#define PKV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes.  Every entry point returns one; nothing is written to any
 * device buffer when a call returns an error. */
typedef enum {
  PKV_OK = 0,
  PKV_ERR_INVALID_ARGUMENT = -1,  /* null pointer, bad shape, misaligned buffer, buffer too small */
  PKV_ERR_BAD_TAG = -2,           /* a block tag is not a pkv_tag_t value */
  PKV_ERR_PAGE_OUT_OF_RANGE = -3, /* a written row's logical page is past the page table, or its
                                     physical page is < -1 or >= pool_pages */
  PKV_ERR_PAGE_UNMAPPED = -4,     /* a written row's logical page maps to -1 */
  PKV_ERR_PAGE_ALIAS = -5,        /* one physical page written through two (request, logical page) pairs */
  PKV_ERR_OUT_OF_MEMORY = -6,     /* host or device allocation failed */
  PKV_ERR_DEVICE = -7             /* no usable GPU, wrong device, or a HIP call / launch failed */
} pkv_status_t;

/* Per-block precision tag (Eq. 14 tiers; K4V4 is the uniform 4-bit
 * representation of the paper's transport ablation, Section V-C). */
typedef enum {
  PKV_TAG_FP16 = 0, /* keys and values binary16 */
  PKV_TAG_K8V8 = 1, /* 8-bit keys, 8-bit values */
  PKV_TAG_K8V4 = 2, /* 8-bit keys, 4-bit values */
  PKV_TAG_K4V4 = 3  /* 4-bit keys, 4-bit values */
} pkv_tag_t;

typedef enum { PKV_OUT_FP16 = 0, PKV_OUT_BF16 = 1 } pkv_out_dtype_t;

/* Which key channels form a rotary pair (the model-aware RoPE correction of
 * Section IV-D: the Delta rotation of Eq. 3 must use the model's own RoPE).
 * Only the first rotary_dim channels rotate; the rest pass through.
 *   PKV_ROPE_HALF:        pair (i, i + rotary_dim/2), i < rotary_dim/2 (Llama, Qwen, NeoX);
 *   PKV_ROPE_INTERLEAVED: pair (2i, 2i + 1), i < rotary_dim/2 (GPT-J, GLM).
 * Pair i turns by Delta * f_i with f_i = inv_freq[i], or rope_theta^(-2i/rotary_dim)
 * when inv_freq is NULL. */
typedef enum { PKV_ROPE_HALF = 0, PKV_ROPE_INTERLEAVED = 1 } pkv_rope_style_t;

/* Paged KV cache layout (see "caches" above).  PKV_KV_PAIRED keeps a page's K
 * and V slots in one contiguous run; on MI355X the restore writes it 5-7%
 * faster than two separate caches. */
typedef enum { PKV_KV_SEPARATE = 0, PKV_KV_PAIRED = 1 } pkv_kv_layout_t;

/* Model and cache geometry, shared by all requests of a plan.
 * Constraints (else PKV_ERR_INVALID_ARGUMENT):
 *   num_layers >= 1; 1 <= num_kv_heads; head_dim % 16 == 0, 16 <= head_dim <= 512;
 *   num_kv_heads * head_dim <= 4096; 1 <= block_tokens <= 1024;
 *   (block_tokens * num_kv_heads * head_dim) % 32 == 0 (every tile 16-byte aligned);
 *   page_size a power of two in [1, 2^20], one page of one cache at most 2 GiB
 *   (page_size * num_kv_heads * head_dim * 2 <= 2^31 bytes); pool_pages >= 1;
 *   rope_theta finite and > 0; out_dtype a pkv_out_dtype_t value;
 *   rope_style a pkv_rope_style_t value; rotary_dim 0 (= head_dim) or a
 *   multiple of 16 in [16, head_dim]; inv_freq NULL or rotary_dim/2 finite
 *   values (copied at plan time); kv_layout a pkv_kv_layout_t value.  A
 *   zero-initialised tail gives full rotate-half RoPE with rope_theta
 *   frequencies and separate caches. */
typedef struct {
  int32_t num_layers;   /* L */
  int32_t num_kv_heads; /* H */
  int32_t head_dim;     /* D */
  int32_t block_tokens; /* B: tokens per checkpoint block (the repair/reuse unit of Eq. 12) */
  int32_t page_size;    /* P: token slots per KV page */
  int32_t out_dtype;    /* pkv_out_dtype_t of k_cache / v_cache */
  int64_t pool_pages;   /* pages per layer in each cache */
  double rope_theta;    /* RoPE base */
  int32_t rope_style;   /* pkv_rope_style_t */
  int32_t rotary_dim;   /* rotated channels per head; 0 = head_dim */
  const double* inv_freq; /* host [rotary_dim/2] pair frequencies, or NULL for rope_theta^(-2i/rotary_dim) */
  int32_t kv_layout;      /* pkv_kv_layout_t */
  int32_t reserved;       /* must be 0 */
} pkv_model_t;

/* One resumed request (one aligned suffix S).  Host arrays are copied by
 * pkv_restore_plan; the caller may free them when it returns. */
typedef struct {
  int32_t suffix_tokens;       /* N = |S| >= 0; NB = ceil(N / B) blocks, the last may be partial */
  int32_t delta;               /* Delta = rho_i - omega_i (new minus old position), the same for all of S */
  int64_t dst_row0;            /* rho_0 >= 0: logical destination row of suffix token 0 */
  const uint8_t* tags;         /* host [NB] pkv_tag_t (may be NULL when N == 0) */
  const uint8_t* repair_mask;  /* host [NB], nonzero = block in R (skipped, its payload never read) */
  const int32_t* page_table;   /* host [num_logical_pages], physical page or -1 = unmapped */
  int32_t num_logical_pages;   /* >= 0 */
  int32_t reserved;            /* must be 0 */
  uint64_t payload_offset;     /* byte offset of this request's checkpoint in `payload`; % 16 == 0 */
  uint64_t scale_offset;       /* binary16-element offset of its scales in `scales`; % 4 == 0 */
} pkv_request_t;

typedef struct pkv_plan pkv_plan_t; /* opaque, immutable once built */

/* Sizes of one request's checkpoint: payload bytes and binary16 scale
 * elements (layout above).  Host only, no GPU needed.  Validates the model
 * and the tags. */
pkv_status_t pkv_payload_size(const pkv_model_t* model, const pkv_request_t* request,
                              uint64_t* payload_bytes, uint64_t* scale_elems);

/* Validate a resume and build its plan on the current HIP device.
 *   model, requests[0..num_requests) : as above (num_requests >= 0; 0 gives an empty plan);
 *   out                              : receives the plan (set to NULL on error).
 * All validation runs on the host before any HIP call (so every argument
 * error is reported without a GPU): shapes, tags, reserved fields, offset
 * alignment, every page touched by a row of a reused block (mapped, in
 * range) and page ownership (no physical page written through two
 * (request, logical page) pairs).  Then the tile list, per-request page
 * tables and cos/sin(Delta * theta_i) tables (computed in double precision
 * on the host) are copied to device memory owned by the plan (synchronous).
 * Errors: any status above. */
pkv_status_t pkv_restore_plan(const pkv_model_t* model, const pkv_request_t* requests, int32_t num_requests,
                              pkv_plan_t** out);

/* Enqueue the restore described by `plan` on `hip_stream` (a hipStream_t;
 * NULL = the default stream) and return without waiting.
 *   payload      : >= the plan's payload_bytes (pkv_plan_query), 16-byte aligned;
 *   scales       : binary16, >= the plan's scale_bytes, 8-byte aligned;
 *     either may be device memory or pinned host memory (hipHostMalloc,
 *     which is mapped for the device): the kernel then reads the checkpoint
 *     over the host link (a zero-copy restore: only the reused blocks'
 *     bytes cross it, in one launch).  Pageable host memory and another
 *     device's memory are PKV_ERR_INVALID_ARGUMENT;
 *   k_cache/v_cache : device memory of the plan's device, 16-byte aligned, not
 *                  overlapping the inputs.  PKV_KV_SEPARATE: two buffers of
 *                  cache_bytes each (>= L*pool_pages*P*H*D*2), not overlapping
 *                  each other.  PKV_KV_PAIRED: one buffer of cache_bytes
 *                  (>= 2*L*pool_pages*P*H*D*2) starting at k_cache, with
 *                  v_cache = k_cache + P*H*D*2 bytes;
 *   *_bytes      : the caller's allocation sizes, checked against what the plan reads / writes.
 * The current device must be the plan's device.  All buffers must stay alive
 * until the stream has passed the restore.  Calls that share a plan are safe
 * concurrently only on disjoint caches.  Errors: PKV_ERR_INVALID_ARGUMENT,
 * PKV_ERR_DEVICE (launch failure; asynchronous faults surface at the next
 * synchronisation of the stream).  The call enqueues one kernel and allocates
 * nothing, so it may be captured in a HIP graph; the checks above then run
 * once, at capture, and every replay uses the captured pointers. */
pkv_status_t pkv_restore(const pkv_plan_t* plan, const void* payload, uint64_t payload_bytes, const void* scales,
                         uint64_t scale_bytes, void* k_cache, void* v_cache, uint64_t cache_bytes, void* hip_stream);

/* Streamed restore from host memory (the transport of Section IV-D and
 * Section V-A: the checkpoint sits in CPU DRAM, copies are asynchronous from
 * pinned memory, and only reused blocks move).  For each layer in turn, the
 * byte ranges of that layer's reused (F) blocks and that layer's scale
 * entries are copied host -> device, into `payload` / `scales` at the
 * checkpoint's own offsets, on copy streams owned by the plan; the layer's
 * restore is then enqueued on `hip_stream` behind those copies.  Copies of
 * layer l + 1 therefore overlap the restore of layer l.  Repair-block
 * payload bytes cross the host link only where a repair block sits between
 * two reused ones closer than 512 KiB apart (one copy then covers all three:
 * cheaper than a second copy's setup); a layer's scale entries, 8 bytes per
 * block and head, are copied whole.  The copies start only after work already
 * enqueued on `hip_stream` (which may still read `payload`) has finished.
 *   host_payload / host_scales : host memory holding the whole checkpoint
 *     (>= the plan's payload_bytes / scale_bytes).  Pinned memory
 *     (hipHostMalloc) gives asynchronous copies at link speed; pageable
 *     memory works, but the runtime stages it and the call may block.
 *   payload / scales : device buffers receiving the copies (as in
 *     pkv_restore); bytes outside the copied ranges are not written.
 *   k_cache, v_cache, cache_bytes, hip_stream : as in pkv_restore.
 * Returns after enqueueing; everything is complete once `hip_stream` has
 * passed the last layer.  The host buffers must stay valid until then.
 * Calls on one plan share its copy streams and events, so they must not
 * overlap: not from two host threads at once, and a call on another stream
 * must wait until the earlier call's work has finished (successive calls on
 * one stream are ordered by it).  The plan must be a restore plan.  The
 * streams and events are created on the first call and released by
 * pkv_free.  Errors: PKV_ERR_INVALID_ARGUMENT,
 * PKV_ERR_DEVICE. */
pkv_status_t pkv_restore_from_host(const pkv_plan_t* plan, const void* host_payload, uint64_t host_payload_bytes,
                                   const void* host_scales, uint64_t host_scale_bytes, void* payload,
                                   uint64_t payload_bytes, void* scales, uint64_t scale_bytes, void* k_cache,
                                   void* v_cache, uint64_t cache_bytes, void* hip_stream);

/* The streamed restore of pkv_restore_from_host for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): no device checkpoint buffers are passed,
 * and the call allocates nothing.  The checkpoint is staged through a buffer
 * of the library, a static device array of 64 MiB (payload windows) + 4 MiB
 * (scales) that each GPU the library runs on holds until the process ends.
 * For each layer and request in turn, on `hip_stream` only: the request's
 * layer scales are copied into the stage, then the request's reused blocks
 * (payload order) go through in windows of at most 64 MiB, each copied from
 * host memory (blocks closer than 512 KiB merged into one copy) and restored
 * before the next window's copies start.  One DMA stream carries every copy,
 * so the host link runs below the two-stream rate of pkv_restore_from_host.
 *   host_payload / host_scales : pinned host memory (hipHostMalloc) holding
 *     the whole checkpoint (>= the plan's payload_bytes / scale_bytes);
 *     pageable memory is PKV_ERR_INVALID_ARGUMENT;
 *   k_cache, v_cache, cache_bytes, hip_stream : as in pkv_restore.
 * Limit: one request-layer's scales, ceil(N / B) * H * 8 bytes, must fit in
 * 4 MiB (PKV_ERR_INVALID_ARGUMENT otherwise, before anything is enqueued);
 * every block fits a window.  Every call on one GPU shares that GPU's stage
 * and leaves the last window in it (nothing in it needs to start at zero):
 * calls that overlap on one GPU -- on different streams, or from several
 * threads -- race and must be ordered by the caller.  Returns after
 * enqueueing.  Errors: PKV_ERR_INVALID_ARGUMENT, PKV_ERR_DEVICE. */
pkv_status_t pkv_restore_from_host_noalloc(const pkv_plan_t* plan, const void* host_payload,
                                           uint64_t host_payload_bytes, const void* host_scales,
                                           uint64_t host_scale_bytes, void* k_cache, void* v_cache,
                                           uint64_t cache_bytes, void* hip_stream);

/* Release a plan and its device memory.  NULL is a no-op.  The caller must
 * make sure no enqueued restore still uses it. */
void pkv_free(pkv_plan_t* plan);

/* ----------------------------------------------------------------------------
 * Checkpoint write (the offload side, Section IV-D): quantize-and-gather.
 *
 * Reads every block of each request's suffix from the OLD context's paged
 * caches (k_cache / v_cache in model->kv_layout, of model->out_dtype)
 * and writes the checkpoint in the format above, which pkv_restore reads:
 *   FP16 tag: the binary16 value nearest (round to nearest even) to each
 *     cache value; 8/4-bit tags, per (layer, block, head, K|V) over the valid
 *     rows: zero = the largest binary16 <= min, scale = the smallest binary16
 *     >= (max - zero)/(2^bits - 1), code = round-half-even((x - zero)/scale)
 *     clipped to [0, 2^bits - 1] (code 0 when the scale is 0), so every value
 *     decodes within scale/2.  Padding rows of a partial last block are
 *     written as code 0 / +0.  Scale entries of FP16 blocks are written 0.
 *   Values must be finite, and within the binary16 range (|x| <= 65504) for
 *     quantized tags, so that zero and scale are binary16 numbers.
 * The repair set is not known when a checkpoint is written, so every block
 * is encoded.
 * ---------------------------------------------------------------------------- */
typedef struct {
  int32_t suffix_tokens;      /* N >= 0 */
  int32_t reserved;           /* must be 0 */
  int64_t src_row0;           /* omega_0 >= 0: old logical row of suffix token 0 */
  const uint8_t* tags;        /* host [NB] pkv_tag_t (frozen per-block precision tags) */
  const int32_t* page_table;  /* host [num_logical_pages] of the old context, -1 = unmapped */
  int32_t num_logical_pages;  /* >= 0 */
  int32_t reserved2;          /* must be 0 */
  uint64_t payload_offset;    /* bytes, % 16 == 0; request payload ranges must not overlap */
  uint64_t scale_offset;      /* binary16 elements, % 4 == 0; request scale ranges must not overlap */
} pkv_checkpoint_request_t;

/* Validate a checkpoint write and build its plan on the current HIP device
 * (same model constraints as pkv_restore_plan).  Every row of every block must sit
 * on a mapped, in-range page (PKV_ERR_PAGE_UNMAPPED / _OUT_OF_RANGE);
 * overlapping payload or scale ranges of two requests are
 * PKV_ERR_INVALID_ARGUMENT.  Host arrays are copied.  Errors: as
 * pkv_restore_plan. */
pkv_status_t pkv_checkpoint_plan(const pkv_model_t* model, const pkv_checkpoint_request_t* requests,
                                 int32_t num_requests, pkv_plan_t** out);

/* Enqueue the checkpoint write of a pkv_checkpoint_plan on `hip_stream`.
 *   k_cache / v_cache : device memory of the plan's device, read only, 16-byte
 *                       aligned, cache_bytes as in pkv_restore for the model's kv_layout;
 *   payload / scales  : outputs, >= the plan's payload_bytes / scale_bytes,
 *                       16- / 8-byte aligned, not overlapping each other or the
 *                       caches: device memory of the plan's device, or pinned
 *                       host memory (hipHostMalloc), which the kernel writes
 *                       over the host link (the checkpoint lands in CPU DRAM,
 *                       where the paper keeps it, with no staging copy).
 * Pageable host memory or another device's memory, for any buffer, is
 * PKV_ERR_INVALID_ARGUMENT, and nothing is written.
 * Only bytes inside the requests' checkpoint ranges are written.
 * A restore plan passed here (or a checkpoint plan passed to pkv_restore) is
 * PKV_ERR_INVALID_ARGUMENT.  Errors: PKV_ERR_INVALID_ARGUMENT, PKV_ERR_DEVICE.
 * Like pkv_restore, it enqueues one kernel, allocates nothing and may be
 * captured in a HIP graph. */
pkv_status_t pkv_quantize_gather(const pkv_plan_t* plan, const void* k_cache, const void* v_cache,
                                 uint64_t cache_bytes, void* payload, uint64_t payload_bytes, void* scales,
                                 uint64_t scale_bytes, void* hip_stream);

/* ----------------------------------------------------------------------------
 * Resume planner (Section IV-B, Eq. 9, 11, 12): the block-aligned repair set
 * R of one request, as the repair_mask a pkv_request_t takes.  Host only.
 *   D = { i in S : i < min(dirty_tokens, N) }        (Eq. 9; token i of S is
 *       i tokens past the edit, and dirty_tokens is the length model's
 *       prediction d_hat, computed elsewhere);
 *   H = the k highest importance[i] over i in S \ D  (Eq. 11), with
 *       k = floor(kappa * |S \ D| + 1/2) in double precision and ties
 *       broken toward the smaller i;
 *   R = the blocks of B tokens that meet D u H, F = the rest (Eq. 12).
 *   suffix_tokens  : N >= 0;  block_tokens : B, 1 <= B <= 1024;
 *   dirty_tokens   : d_hat >= 0 (values past N mean all of S);
 *   importance     : host [N] stored scores I_i(0), finite (may be NULL when N == 0);
 *   kappa          : the nonlocal budget fraction, 0 <= kappa <= 1;
 *   repair_mask    : host [ceil(N / B)] output, 1 = block in R, 0 = in F;
 *   nonlocal_tokens: output |H| (may be NULL).
 * Errors: PKV_ERR_INVALID_ARGUMENT, PKV_ERR_OUT_OF_MEMORY. */
pkv_status_t pkv_plan_repair(int32_t suffix_tokens, int32_t block_tokens, int64_t dirty_tokens,
                             const float* importance, double kappa, uint8_t* repair_mask, int64_t* nonlocal_tokens);

/* What a plan reads and writes (for sizing buffers and for bandwidth
 * accounting).  For a checkpoint plan, bytes_read counts cache rows read and
 * bytes_written the payload and scale bytes written; restored_rows counts the
 * suffix rows encoded per cache. */
typedef struct {
  int64_t num_requests;
  int64_t num_units;          /* work items: restore plans, the part of a reused block of one layer inside one
                                 cache page (one workgroup each); checkpoint plans, (request, layer, block) */
  int64_t restored_rows;      /* token rows written per cache, summed over layers and requests */
  uint64_t payload_bytes;     /* bytes of `payload` the plan may touch (max over requests of offset + size) */
  uint64_t scale_bytes;       /* bytes of `scales` likewise */
  uint64_t cache_bytes;       /* bytes of each cache (PKV_KV_SEPARATE) or of the one paired cache */
  uint64_t bytes_read;        /* payload + scale bytes of reused blocks (what the restore must read) */
  uint64_t bytes_written;     /* output bytes, K and V */
  int32_t device;             /* HIP device the plan lives on */
  int32_t kind;               /* 0 = restore plan, 1 = checkpoint plan */
  uint64_t host_copy_bytes;   /* restore plans: bytes pkv_restore_from_host copies (F-block ranges + scales) */
  int64_t host_copies;        /* restore plans: number of host -> device copies it issues (after chunking) */
} pkv_plan_info_t;

pkv_status_t pkv_plan_query(const pkv_plan_t* plan, pkv_plan_info_t* info);

/* Bytes of request `req`'s checkpoint payload, all layers (the clustered
 * layout above, repair blocks included), for a restore or a checkpoint plan:
 * the payload that Section IV-D's quantize-and-gather writes and its
 * transport stage draws F blocks from (Eq. 12), and the per-representation
 * checkpoint size of Section V-D.  Host only.  Errors:
 * PKV_ERR_INVALID_ARGUMENT (NULL plan or bytes, req outside [0, num_requests)). */
pkv_status_t pkv_plan_payload_bytes(const pkv_plan_t* plan, int32_t req, uint64_t* bytes);

/* Static description of a status code. */
const char* pkv_status_string(pkv_status_t status);

#ifdef __cplusplus
}
#endif

#endif /* PKV_H */
