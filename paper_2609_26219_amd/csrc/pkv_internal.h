// Internal structures shared by the host plan builder and the device kernel.
#ifndef PKV_INTERNAL_H
#define PKV_INTERNAL_H

#include <stdint.h>

#include <vector>

#include "pkv.h"

namespace pkv {

constexpr int kMaxHeadDim = 512;
constexpr int kMaxRowElems = 4096;   // num_kv_heads * head_dim
constexpr int kMaxBlockTokens = 1024;
constexpr int kWorkgroup = 256;       // threads per workgroup

// Key / value bits per channel of each tag (Eq. 14 tiers plus uniform 4-bit).
constexpr int kKeyBits[4] = {16, 8, 8, 4};
constexpr int kValueBits[4] = {16, 8, 4, 4};

// One workgroup's work: every head of one reused block of one layer of one
// request.  48 bytes.
struct Unit {
  uint64_t k_off;      // byte offset of the block's K tile in the payload
  uint64_t v_off;      // byte offset of its V tile
  uint64_t scale_off;  // binary16-element offset of its (head 0, K, scale) entry
  int64_t row0;        // logical destination row of the block's first token
  int32_t layer;
  int32_t req;
  int32_t tag;
  int32_t n_valid;     // valid tokens in the block (< B only for the last block)
};
static_assert(sizeof(Unit) == 48, "Unit layout");

// Per-request device metadata.  32 bytes.
struct ReqDev {
  int64_t table_off;  // offset, in doubles, of the request's [D/2][2] (cos, sin) table
  int64_t pt_off;     // offset, in int32, of the request's page table
  int32_t rotate;     // Delta != 0
  int32_t num_logical_pages;
  int64_t reserved;
};
static_assert(sizeof(ReqDev) == 32, "ReqDev layout");

// Everything the plan needs on the device, built on the host.
struct HostPlan {
  pkv_model_t model;
  std::vector<Unit> units;
  std::vector<ReqDev> reqs;
  std::vector<double> tables;      // per request [D/2][2]
  std::vector<int32_t> page_tables;
  pkv_plan_info_t info;
  int32_t log2_page;
};

// Validate and build the host side of a plan.  Makes no HIP call.
pkv_status_t build_host_plan(const pkv_model_t* model, const pkv_request_t* requests, int32_t num_requests,
                             HostPlan* out);

// Bytes of one layer of a request's checkpoint (tags already validated).
uint64_t layer_payload_bytes(const pkv_model_t& m, const uint8_t* tags, int64_t nb);

}  // namespace pkv

#endif  // PKV_INTERNAL_H
