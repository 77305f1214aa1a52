// Internal structures shared by the host plan builder and the device kernel.
#ifndef PKV_INTERNAL_H
#define PKV_INTERNAL_H

#include <stdint.h>

#include <vector>

#include "pkv.h"

namespace pkv {

constexpr int kMaxHeadDim = 512;

// The hardware deals a launch's workgroups to the eight XCDs in turn
// (workgroup b runs on XCD b % 8), each XCD with its own L2.  Kernels take
// their work item from xcd_grouped(b, grid), which renumbers the workgroups
// so that kXcdGroup consecutive work items run on one XCD and share its L2
// (neighbouring payload tiles, scale lines, work items).  It is a permutation
// of [0, grid); the last, partial round of 8 * kXcdGroup keeps its order.
constexpr int64_t kXcdCount = 8;
constexpr int64_t kXcdGroup = 8;
constexpr int64_t xcd_grouped(int64_t b, int64_t grid) {
  const int64_t round = kXcdCount * kXcdGroup;
  if (b >= grid / round * round) return b;
  const int64_t slot = b / kXcdCount;
  return slot / kXcdGroup * round + (b % kXcdCount) * kXcdGroup + slot % kXcdGroup;
}
constexpr int kMaxRowElems = 4096;   // num_kv_heads * head_dim
constexpr int kMaxBlockTokens = 1024;
constexpr int kWorkgroup = 256;       // threads per workgroup
// Target output per unit: units of about 16K elements per cache (32 KiB of
// binary16/bfloat16) keep workgroups short, so the launch drains evenly.
constexpr int kUnitElems = 16384;

// Key / value bits per channel of each tag (Eq. 14 tiers plus uniform 4-bit).
constexpr int kKeyBits[4] = {16, 8, 8, 4};
constexpr int kValueBits[4] = {16, 8, 4, 4};

// One work item.  Restore: every head of up to `n_valid` consecutive tokens
// of one reused block of one layer of one request.  Checkpoint write: one
// whole block of one layer of one request.  64 bytes.
struct Unit {
  uint64_t k_off;      // byte offset of the unit's first K row in the payload
  uint64_t v_off;      // byte offset of its first V row
  uint64_t scale_off;  // binary16-element offset of the block's (head 0, K, scale) entry
  int64_t row0;        // logical row of the unit's first token (destination / old context)
  int64_t pt_off;      // offset, in int32, of the request's page table
  union {
    int32_t table_off;  // restore: offset, in doubles, of the request's [D/2][2] (cos, sin) table
    int32_t page0;      // checkpoint: physical page of logical page row0 >> log2(P)
  };
  int32_t layer;
  int32_t tag;         // bits 0-7: pkv_tag_t; bit 8: rotate keys (Delta != 0)
  int32_t n_valid;     // tokens in the unit
  int32_t page1;       // checkpoint: the next two physical pages of the block's rows, -1 past its
  int32_t page2;       //   last page; restore: page1 = the one physical page of the unit's rows, page2 = 0
};
static_assert(sizeof(Unit) == 64, "Unit layout");
constexpr int32_t kUnitRotate = 1 << 8;

// Per-request metadata kept on the host.
struct ReqInfo {
  int64_t table_off;  // offset, in doubles, of the request's table
  int64_t pt_off;     // offset, in int32, of the request's page table
};

struct CopyRange {
  uint64_t off, len;  // bytes
};
// Streamed restore: two copies of one layer whose ranges are at most this
// many bytes apart are merged into one (the repair blocks between them are
// copied too): one host -> device copy costs a fixed setup time that a gap
// of this size takes to transfer at link speed.
#ifndef PKV_HOST_GAP_BYTES
#define PKV_HOST_GAP_BYTES (512u << 10)
#endif
constexpr uint64_t kHostGapBytes = PKV_HOST_GAP_BYTES;
// Streamed restore: copy streams that copy chunks are dealt to.
#ifndef PKV_HOST_COPY_STREAMS
#define PKV_HOST_COPY_STREAMS 2
#endif
constexpr int kHostCopyStreams = PKV_HOST_COPY_STREAMS;
static_assert(kHostCopyStreams >= 1 && kHostCopyStreams <= 32, "copy streams are tracked in a 32-bit mask");
// Streamed restore: copies are cut into chunks of at most this many bytes,
// dealt to the copy streams in turn.  One DMA stream alone moves ~40 GB/s;
// two busy together fill the host link (~57 GB/s).  Measured on the
// 8B-shaped 32-layer checkpoint: 16 MiB chunks on two streams 16.8 ms
// (uniform 4-bit) and 31.7 ms (mixed tags), against 33.2 / 33.0 ms with one
// stream and unchunked copies; 4 MiB chunks or four streams were no better.
#ifndef PKV_HOST_CHUNK_BYTES
#define PKV_HOST_CHUNK_BYTES (16ull << 20)
#endif
constexpr uint64_t kHostChunkBytes = PKV_HOST_CHUNK_BYTES;

// The allocation-free streamed restore stages the checkpoint through a
// static device buffer: payload windows in its first kStagePayloadBytes, one
// request-layer's scales in the kStageScaleBytes after them.
constexpr uint64_t kStagePayloadBytes = 64ull << 20;
constexpr uint64_t kStageScaleBytes = 4ull << 20;

// One step of that restore, all on the caller's stream: copy the step's
// scales (if any) and payload ranges from host memory into the stage, then
// restore units [u0, u1) -- one layer of one request -- whose K rows start in
// payload bytes [win_lo, win_hi).  A window holds the most consecutive reused
// blocks, in payload order, that span at most kStagePayloadBytes; payload
// byte o of the window sits at stage offset o - win_lo.
struct StageStep {
  int64_t u0, u1;
  uint64_t win_lo, win_hi;  // absolute payload bytes
  uint64_t scale0;          // absolute binary16 element of the request-layer's scales
  uint64_t scale_elems;     // elements staged before this step (0: none; the stage already holds them)
  int64_t copy0, copy1;     // its payload copies in HostPlan::stage_copies
};
struct StageCopy {
  uint64_t src;  // absolute payload byte offset
  uint64_t dst;  // byte offset into the stage
  uint64_t len;
};

// Everything the plan needs on the device, built on the host.
struct HostPlan {
  int32_t kind = 0;  // 0 = restore, 1 = checkpoint write
  int32_t workgroup = kWorkgroup;
  pkv_model_t model;
  std::vector<Unit> units;
  std::vector<ReqInfo> reqs;
  std::vector<double> tables;      // per request [D/2][2]
  std::vector<int32_t> page_tables;
  pkv_plan_info_t info;
  int32_t log2_page;
  // Restore plans: units are layer-major; layer l owns units
  // [layer_units[l], layer_units[l + 1]).  Host -> device copy ranges of the
  // streamed restore, merged, layer-major: payload bytes and scale bytes,
  // layer l owning [*_layer[l], *_layer[l + 1]).  Kept on the host.
  std::vector<int64_t> layer_units;
  std::vector<CopyRange> payload_ranges, scale_ranges;
  std::vector<int64_t> payload_layer, scale_layer;
  int64_t rotated_rows = 0;  // restore plans: restored rows whose keys rotate (shift != 0)
  std::vector<uint64_t> req_payload_bytes;  // per request: bytes of its checkpoint payload, all layers
  // Restore plans: the schedule of the restore staged through the library's
  // static buffer (add_stage_steps in plan.cpp), or stage_ok = false when a
  // request-layer's scales do not fit it.
  std::vector<StageStep> stage_steps;
  std::vector<StageCopy> stage_copies;
  bool stage_ok = false;
};

// Restore workgroups resident per compute unit, chosen per plan: 8 to 16
// waves (for 4-wave workgroups two to four, one wave per SIMD each; 16 waves
// is the register limit).  Measured on the 8B-shaped 32-layer restore,
// destination rows 7 slots into a page (units of 9, 16 and 7 tokens), us at
// 2 / 3 / 4 workgroups per CU, paired pages:
//   FP16 (read:write 1.00)  1200-1208 / 1233-1248 / 1240-1250
//   K8V8 (0.50)              889-892 /  915-916 /  956-958
//   mixed (0.47)             906-953 /  905-913 /  941-952
//   K8V4 (0.38)              861-867 /  836-837 /  884-885
//   K4V4 (0.25)              874-875 /      780 /  806-816
// separate caches:
//   FP16 1311-1325 / 1333-1347 / 1333-1349, K8V8 963 / 1041 / 1050-1053,
//   mixed 973-991 / 1015-1030 / 1039-1046, K8V4 907-908 / 954-957 / 979-980,
//   K4V4 895-896 / 851-856 / 896-899;
// and with page-aligned rows (16-token units), paired: mixed 891-898 /
// 952-961 / 965, K4V4 774-776 / 836-837 / 847: the best count falls as units
// grow.  Unshifted plans (no rotation, no table) run best with fewer.  The
// one-head-per-GPU share of the same workload restores in 139 us (16 one-wave
// workgroups) whatever the target, the two-head share in 263 us at 8
// one-wave workgroups and 243 at 12 or 16.
int restore_workgroups_per_cu(const HostPlan& hp);

// Validate and build the host side of a plan.  Makes no HIP call.
pkv_status_t build_host_plan(const pkv_model_t* model, const pkv_request_t* requests, int32_t num_requests,
                             HostPlan* out);

// Same for a checkpoint write (quantize-and-gather).
pkv_status_t build_checkpoint_plan(const pkv_model_t* model, const pkv_checkpoint_request_t* requests,
                                   int32_t num_requests, HostPlan* out);

// Checkpoint kernel: one wave per (head, K|V) tile of a block, at most
// kGatherMaxWaves waves per workgroup; a lane holds up to
// gather_loads_per_chunk(n) 16-byte loads of a tile in registers.
constexpr int kGatherMaxWaves = 16;
// A checkpoint unit carries the block's first three source pages, enough
// for every block when block_tokens <= 2 * page_size + 1.
constexpr int kUnitPages = 3;
int32_t gather_workgroup(const pkv_model_t& m);
inline int gather_loads_per_chunk(int nload) { return nload <= 2 ? 2 : nload <= 4 ? 4 : nload <= 8 ? 8 : 16; }

// The plan object behind pkv_plan_t (host metadata + one device allocation).
}  // namespace pkv
struct pkv_plan {
  pkv::HostPlan host;  // units, tables and page tables are dropped after upload
  void* device_mem = nullptr;
  pkv::Unit* d_units = nullptr;
  double* d_tables = nullptr;
  int32_t* d_page_tables = nullptr;
  int device = -1;
  // Dynamic LDS bytes per restore workgroup, sized so that at most
  // restore_workgroups_per_cu() workgroups are resident on a compute unit.
  uint32_t restore_lds = 0;
  // Restore launches of at most this many units (a few rounds of compute
  // units x restore_workgroups_per_cu() resident workgroups; every launch for
  // rows narrow enough for workgroups under kWorkgroup threads) take the late
  // start order of the restore kernel; 0 when the device could not be queried.
  int64_t restore_late_units = 0;
  // Streamed restore: copy streams and events (hipStream_t / hipEvent_t),
  // created on first use.  events[0] marks the caller's stream at entry;
  // events[1 + l * n + k] the end of layer l's chunks on copy stream k.
  std::vector<void*> copy_streams;
  std::vector<void*> events;
};
namespace pkv {
// Copy a built host plan to device memory on the current device and wrap it.
pkv_status_t upload_plan(HostPlan&& hp, pkv_plan** out);

// Bytes of one layer of a request's checkpoint (tags already validated).
uint64_t layer_payload_bytes(const pkv_model_t& m, const uint8_t* tags, int64_t nb);

// Tokens per unit for a model: about kUnitElems output elements, at most one block.
int32_t unit_tokens(const pkv_model_t& m);
int32_t restore_workgroup(const pkv_model_t& m);

// Cache geometry by layout.  A page's slots start at page << page_shift slot
// rows from the layer's start (log2 P, plus one when a page holds its K and V
// slots back to back); a layer spans layer_elems elements of either cache.
int32_t page_shift(const pkv_model_t& m);
int64_t layer_elems(const pkv_model_t& m);
uint64_t cache_bytes(const pkv_model_t& m);  // of each separate cache, or of the paired one

// The cache pointers of a call against the model's layout: both 16-byte
// aligned; separate caches of cache_bytes each must not overlap; a paired
// cache has v_cache = k_cache + P*H*D elements.  `ranges` receives the byte
// ranges the caches occupy (two, or one for a paired cache) for overlap
// checks against other buffers; returns false on a bad placement.
struct ByteRange {
  const void* p;
  uint64_t n;
};
bool cache_ranges(const pkv_model_t& m, const void* k_cache, const void* v_cache, uint64_t bytes, ByteRange (&ranges)[2],
                  int& count);

// What kind of memory a kernel argument is (hipPointerGetAttributes), so that
// no launch ever gets a pointer the kernel would fault on.
//   kernel_accessible: device or managed memory of the plan's device as is,
//     or pinned host memory through its device mapping (*out receives the
//     address the kernel uses); pageable host memory or another device's
//     memory is PKV_ERR_INVALID_ARGUMENT.
//   device_resident: device or managed memory of the plan's device only.
pkv_status_t kernel_accessible(const pkv_plan* plan, const void* p, const void** out);
pkv_status_t device_resident(const pkv_plan* plan, const void* p);

}  // namespace pkv

#endif  // PKV_INTERNAL_H
