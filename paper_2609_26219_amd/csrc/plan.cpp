// Host half of libpkv: argument validation, the checkpoint layout, the work
// list and the RoPE correction tables.  Pure C++ (no HIP calls), so every
// validation path runs without a GPU.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <limits>
#include <new>
#include <tuple>
#include <vector>

#include "pkv.h"
#include "pkv_internal.h"

namespace pkv {
namespace {

bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

int ilog2(int64_t x) {
  int r = 0;
  while ((int64_t(1) << r) < x) ++r;
  return r;
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

pkv_status_t check_model(const pkv_model_t* m) {
  if (!m) return PKV_ERR_INVALID_ARGUMENT;
  if (m->num_layers < 1 || m->num_kv_heads < 1) return PKV_ERR_INVALID_ARGUMENT;
  if (m->head_dim < 16 || m->head_dim > kMaxHeadDim || m->head_dim % 16 != 0) return PKV_ERR_INVALID_ARGUMENT;
  if (int64_t(m->num_kv_heads) * m->head_dim > kMaxRowElems) return PKV_ERR_INVALID_ARGUMENT;
  if (m->block_tokens < 1 || m->block_tokens > kMaxBlockTokens) return PKV_ERR_INVALID_ARGUMENT;
  if ((int64_t(m->block_tokens) * m->num_kv_heads * m->head_dim) % 32 != 0) return PKV_ERR_INVALID_ARGUMENT;
  if (!is_pow2(m->page_size) || m->page_size > (1 << 20)) return PKV_ERR_INVALID_ARGUMENT;
  // One page of one cache is at most 2 GiB: the kernels address inside a page with 32-bit offsets.
  if (int64_t(m->page_size) * m->num_kv_heads * m->head_dim * 2 > (int64_t(1) << 31)) return PKV_ERR_INVALID_ARGUMENT;
  if (m->pool_pages < 1) return PKV_ERR_INVALID_ARGUMENT;
  if (!(isfinite(m->rope_theta) && m->rope_theta > 0.0)) return PKV_ERR_INVALID_ARGUMENT;
  if (m->out_dtype != PKV_OUT_FP16 && m->out_dtype != PKV_OUT_BF16) return PKV_ERR_INVALID_ARGUMENT;
  if (m->rope_style != PKV_ROPE_HALF && m->rope_style != PKV_ROPE_INTERLEAVED) return PKV_ERR_INVALID_ARGUMENT;
  if (m->rotary_dim != 0 && (m->rotary_dim < 16 || m->rotary_dim > m->head_dim || m->rotary_dim % 16 != 0))
    return PKV_ERR_INVALID_ARGUMENT;
  if (m->kv_layout != PKV_KV_SEPARATE && m->kv_layout != PKV_KV_PAIRED) return PKV_ERR_INVALID_ARGUMENT;
  if (m->reserved != 0) return PKV_ERR_INVALID_ARGUMENT;
  if (m->inv_freq) {
    const int32_t R = m->rotary_dim ? m->rotary_dim : m->head_dim;
    for (int32_t i = 0; i < R / 2; ++i)
      if (!isfinite(m->inv_freq[i])) return PKV_ERR_INVALID_ARGUMENT;
  }
  // Cache elements per layer and in total must stay far from int64 overflow.
  const double elems = 2.0 * double(m->num_layers) * double(m->pool_pages) * m->page_size * m->num_kv_heads * m->head_dim;
  if (elems > 1e18) return PKV_ERR_INVALID_ARGUMENT;
  return PKV_OK;
}

// RoPE helpers: rotated channels per head, the frequency of pair i, and the
// pair that element e of key piece j rotates (k = 8j + e; -1 = none).
int32_t rotary_dim(const pkv_model_t& m) { return m.rotary_dim ? m.rotary_dim : m.head_dim; }

double rope_frequency(const pkv_model_t& m, int64_t i) {
  const int32_t R = rotary_dim(m);
  return m.inv_freq ? m.inv_freq[i] : pow(m.rope_theta, -2.0 * double(i) / double(R));
}

int64_t rope_table_pair(const pkv_model_t& m, int64_t k) {
  const int64_t D = m.head_dim, R = rotary_dim(m);
  const int64_t j = k / 8, e = k % 8;
  if (m.rope_style == PKV_ROPE_HALF) {
    // Piece j < R/16 holds channels [8j, 8j+8) and [R/2 + 8j, ...): pairs 8j + e.
    return 8 * j < R / 2 ? 8 * j + e : -1;
  }
  // Interleaved: piece j holds channels [8j, 8j+8) (elements 0..3 are its four
  // pairs) and [D/2 + 8j, ...) (elements 4..7); a pair rotates if inside [0, R).
  const int64_t first = e < 4 ? 8 * j : D / 2 + 8 * j;
  return first + 8 <= R ? first / 2 + e % 4 : -1;
}

pkv_status_t check_request_fields(const pkv_request_t& r) {
  if (r.reserved != 0) return PKV_ERR_INVALID_ARGUMENT;
  if (r.suffix_tokens < 0 || r.num_logical_pages < 0 || r.dst_row0 < 0) return PKV_ERR_INVALID_ARGUMENT;
  if (r.dst_row0 > (int64_t(1) << 50)) return PKV_ERR_INVALID_ARGUMENT;
  if (r.suffix_tokens > 0 && (!r.tags || !r.repair_mask)) return PKV_ERR_INVALID_ARGUMENT;
  if (r.num_logical_pages > 0 && !r.page_table) return PKV_ERR_INVALID_ARGUMENT;
  if (r.payload_offset % 16 != 0 || r.scale_offset % 4 != 0) return PKV_ERR_INVALID_ARGUMENT;
  if (r.payload_offset > (uint64_t(1) << 56) || r.scale_offset > (uint64_t(1) << 56)) return PKV_ERR_INVALID_ARGUMENT;
  return PKV_OK;
}

pkv_status_t check_tags(const pkv_request_t& r, int64_t nb) {
  for (int64_t b = 0; b < nb; ++b)
    if (r.tags[b] > PKV_TAG_K4V4) return PKV_ERR_BAD_TAG;
  return PKV_OK;
}

uint64_t tile_bytes(const pkv_model_t& m, int bits) {
  return uint64_t(m.block_tokens) * m.num_kv_heads * m.head_dim * bits / 8;
}

// Steps of the staged restore for the units [u0, u1) of one request-layer:
// windows of the most consecutive reused blocks (payload order, offsets
// relative to layer_base) that span at most kStagePayloadBytes (one block,
// at most 16 MiB, always fits), each with its copies (blocks closer than
// kHostGapBytes merged); the request-layer's scales, if any, go with the
// first window.
void add_stage_steps(HostPlan& hp, const std::vector<CopyRange>& blocks, int64_t u0, int64_t u1, uint64_t layer_base,
                     uint64_t scale0, uint64_t scale_elems) {
  for (size_t i = 0; i < blocks.size();) {
    const uint64_t lo = blocks[i].off;
    size_t j = i + 1;
    while (j < blocks.size() && blocks[j].off + blocks[j].len - lo <= kStagePayloadBytes) ++j;
    StageStep st;
    st.u0 = u0;
    st.u1 = u1;
    st.win_lo = layer_base + lo;
    st.win_hi = layer_base + blocks[j - 1].off + blocks[j - 1].len;
    st.scale0 = scale0;
    st.scale_elems = i == 0 ? scale_elems : 0;
    st.copy0 = int64_t(hp.stage_copies.size());
    for (size_t a = i; a < j;) {
      size_t b = a + 1;
      while (b < j && blocks[b].off - (blocks[b - 1].off + blocks[b - 1].len) <= kHostGapBytes) ++b;
      const uint64_t c0 = blocks[a].off, c1 = blocks[b - 1].off + blocks[b - 1].len;
      hp.stage_copies.push_back(StageCopy{layer_base + c0, c0 - lo, c1 - c0});
      a = b;
    }
    st.copy1 = int64_t(hp.stage_copies.size());
    hp.stage_steps.push_back(st);
    i = j;
  }
}

}  // namespace

int32_t page_shift(const pkv_model_t& m) { return ilog2(m.page_size) + (m.kv_layout == PKV_KV_PAIRED ? 1 : 0); }

int64_t layer_elems(const pkv_model_t& m) {
  return (m.kv_layout == PKV_KV_PAIRED ? 2 : 1) * m.pool_pages * int64_t(m.page_size) * m.num_kv_heads * m.head_dim;
}

uint64_t cache_bytes(const pkv_model_t& m) { return uint64_t(m.num_layers) * uint64_t(layer_elems(m)) * 2; }

bool cache_ranges(const pkv_model_t& m, const void* k_cache, const void* v_cache, uint64_t bytes, ByteRange (&ranges)[2],
                  int& count) {
  const uintptr_t k = reinterpret_cast<uintptr_t>(k_cache), v = reinterpret_cast<uintptr_t>(v_cache);
  if (k % 16 || v % 16) return false;
  if (m.kv_layout == PKV_KV_PAIRED) {
    if (v != k + uint64_t(m.page_size) * m.num_kv_heads * m.head_dim * 2) return false;
    ranges[0] = ByteRange{k_cache, bytes};
    count = 1;
    return true;
  }
  if (k < v + bytes && v < k + bytes) return false;
  ranges[0] = ByteRange{k_cache, bytes};
  ranges[1] = ByteRange{v_cache, bytes};
  count = 2;
  return true;
}

int restore_workgroups_per_cu(const HostPlan& hp) {
  // The memory system streams best with about 32K output elements of work in
  // flight per compute unit (two thirds of that for plans reading half a byte
  // or more per byte written, 1.14x for those reading under 0.3; three
  // quarters for units that do not rotate
  // their keys, and again for separate K and V caches; half again for rows
  // narrow enough to take workgroups under 256 threads): so many units at a
  // time, between 8 and 16 waves' worth (two to four 4-wave workgroups).
  const pkv_plan_info_t& info = hp.info;
  const int waves = std::max(1, hp.workgroup / 64);
  const int lo = std::max(1, 8 / waves), hi = std::max(1, 16 / waves);
  if (info.num_units == 0 || info.bytes_written == 0 || info.restored_rows == 0) return hi;
  const double ratio = double(info.bytes_read) / double(info.bytes_written);
  const double rotated = double(hp.rotated_rows) / double(info.restored_rows);
  const double target =
      32768.0 * (ratio >= 0.49 ? 2.0 / 3.0 : ratio >= 0.3 ? 1.0 : 1.14) * (0.75 + 0.25 * rotated) *
      (hp.model.kv_layout == PKV_KV_SEPARATE ? 0.75 : 1.0) * (hp.workgroup < kWorkgroup ? 1.5 : 1.0);
  const double unit_elems =
      double(info.restored_rows) * hp.model.num_kv_heads * hp.model.head_dim / double(info.num_units);
  const double n = std::floor(target / unit_elems + 0.5);
  return n < lo ? lo : n > hi ? hi : int(n);
}

// Threads of a restore workgroup: enough that each thread owns at most four
// tokens of the largest unit (units stop at page ends), in whole waves, at
// most kWorkgroup.  Rows of 8 heads x 128 keep 256; a one-head row of 128
// takes one wave, so shards with few heads per GPU do not leave most of each
// workgroup idle.
int32_t restore_workgroup(const pkv_model_t& m) {
  const int64_t cols = int64_t(m.num_kv_heads) * m.head_dim / 16;
  const int64_t tokens = std::min<int64_t>(unit_tokens(m), m.page_size);
  const int64_t threads = (cols * ceil_div(tokens, 4) + 63) / 64 * 64;
  return int32_t(std::max<int64_t>(64, std::min<int64_t>(kWorkgroup, threads)));
}

int32_t unit_tokens(const pkv_model_t& m) {
  const int64_t per = kUnitElems / (int64_t(m.num_kv_heads) * m.head_dim);
  return int32_t(std::max<int64_t>(1, std::min<int64_t>(per, m.block_tokens)));
}

uint64_t layer_payload_bytes(const pkv_model_t& m, const uint8_t* tags, int64_t nb) {
  uint64_t total = 0;
  for (int64_t b = 0; b < nb; ++b) total += tile_bytes(m, kKeyBits[tags[b]]) + tile_bytes(m, kValueBits[tags[b]]);
  return total;
}

pkv_status_t build_host_plan(const pkv_model_t* model, const pkv_request_t* requests, int32_t num_requests,
                             HostPlan* out) {
  pkv_status_t st = check_model(model);
  if (st != PKV_OK) return st;
  if (num_requests < 0 || (num_requests > 0 && !requests) || !out) return PKV_ERR_INVALID_ARGUMENT;
  const pkv_model_t& m = *model;
  const int64_t B = m.block_tokens, H = m.num_kv_heads, D = m.head_dim, P = m.page_size, L = m.num_layers;
  const int lp2 = ilog2(P);

  // Field, tag and page checks, request by request.
  for (int32_t r = 0; r < num_requests; ++r) {
    const pkv_request_t& q = requests[r];
    if ((st = check_request_fields(q)) != PKV_OK) return st;
    const int64_t nb = ceil_div(q.suffix_tokens, B);
    if ((st = check_tags(q, nb)) != PKV_OK) return st;
  }
  // Every page touched by a row of a reused block: in range and mapped;
  // collect (physical page, request, logical page) for the ownership check.
  std::vector<std::tuple<int64_t, int32_t, int64_t>> touched;
  for (int32_t r = 0; r < num_requests; ++r) {
    const pkv_request_t& q = requests[r];
    const int64_t nb = ceil_div(q.suffix_tokens, B);
    int64_t last_lp = -1;
    for (int64_t b = 0; b < nb; ++b) {
      if (q.repair_mask[b]) continue;
      const int64_t n_valid = std::min<int64_t>(B, q.suffix_tokens - b * B);
      const int64_t first_row = q.dst_row0 + b * B;
      const int64_t last_row = first_row + n_valid - 1;
      for (int64_t lp = std::max(first_row >> lp2, last_lp + 1); lp <= (last_row >> lp2); ++lp) {
        if (lp >= q.num_logical_pages) return PKV_ERR_PAGE_OUT_OF_RANGE;
        const int32_t pp = q.page_table[lp];
        if (pp == -1) return PKV_ERR_PAGE_UNMAPPED;
        if (pp < -1 || pp >= m.pool_pages) return PKV_ERR_PAGE_OUT_OF_RANGE;
        touched.emplace_back(pp, r, lp);
        last_lp = lp;
      }
    }
  }
  std::sort(touched.begin(), touched.end());
  for (size_t i = 1; i < touched.size(); ++i) {
    if (std::get<0>(touched[i]) == std::get<0>(touched[i - 1]) &&
        (std::get<1>(touched[i]) != std::get<1>(touched[i - 1]) ||
         std::get<2>(touched[i]) != std::get<2>(touched[i - 1])))
      return PKV_ERR_PAGE_ALIAS;
  }

  // Build: tile list, per-request metadata, page tables, cos/sin tables.
  HostPlan& hp = *out;
  hp.model = m;
  hp.log2_page = lp2;
  hp.units.clear();
  hp.reqs.clear();
  hp.tables.clear();
  hp.page_tables.clear();
  memset(&hp.info, 0, sizeof(hp.info));
  hp.info.num_requests = num_requests;
  hp.info.cache_bytes = cache_bytes(m);

  if (int64_t(num_requests) * D > std::numeric_limits<int32_t>::max()) return PKV_ERR_INVALID_ARGUMENT;
  try {
    hp.reqs.resize(num_requests);
    hp.req_payload_bytes.assign(size_t(num_requests), 0);
    hp.stage_steps.clear();
    hp.stage_copies.clear();
    hp.tables.resize(size_t(num_requests) * size_t(D));
    // Per request: page table, cos/sin table, block offsets inside a layer.
    std::vector<std::vector<uint64_t>> block_off(num_requests);
    std::vector<uint64_t> layer_bytes(num_requests, 0);
    for (int32_t r = 0; r < num_requests; ++r) {
      const pkv_request_t& q = requests[r];
      const int64_t nb = ceil_div(q.suffix_tokens, B);
      ReqInfo& rd = hp.reqs[r];
      rd.table_off = int64_t(r) * D;
      rd.pt_off = int64_t(hp.page_tables.size());
      hp.page_tables.insert(hp.page_tables.end(), q.page_table, q.page_table + q.num_logical_pages);
      // cos / sin of Delta * f_i in double precision, laid out in the
      // kernel's element order: entry 8j + e is the pair that element e of
      // key piece j rotates (rope_table_pair); pass-through entries are (1, 0).
      for (int64_t k = 0; k < D / 2; ++k) {
        const int64_t i = rope_table_pair(m, k);
        const double ang = i >= 0 ? double(q.delta) * rope_frequency(m, i) : 0.0;
        hp.tables[size_t(r) * D + 2 * k] = q.delta && i >= 0 ? cos(ang) : 1.0;
        hp.tables[size_t(r) * D + 2 * k + 1] = q.delta && i >= 0 ? sin(ang) : 0.0;
      }
      if (nb == 0) continue;
      // Block offsets inside one layer: runs by tag, ascending blocks.
      block_off[r].resize(nb);
      uint64_t pos = 0;
      for (int tag = 0; tag < 4; ++tag)
        for (int64_t b = 0; b < nb; ++b)
          if (q.tags[b] == tag) {
            block_off[r][b] = pos;
            pos += tile_bytes(m, kKeyBits[tag]) + tile_bytes(m, kValueBits[tag]);
          }
      layer_bytes[r] = pos;
      hp.req_payload_bytes[r] = uint64_t(L) * pos;
      hp.info.payload_bytes = std::max<uint64_t>(hp.info.payload_bytes, q.payload_offset + uint64_t(L) * pos);
      hp.info.scale_bytes =
          std::max<uint64_t>(hp.info.scale_bytes, (q.scale_offset + uint64_t(L) * nb * H * 4) * 2);
    }
    // Work list, layer-major, and the streamed restore's copy ranges.
    const int64_t per_unit = unit_tokens(m);
    hp.workgroup = restore_workgroup(m);
    // Append a copy, merging it with the previous one (if that one is at
    // index >= first) when it starts at most `gap` bytes after that one ends.
    auto add_range = [](std::vector<CopyRange>& v, int64_t first, uint64_t off, uint64_t len, uint64_t gap) {
      if (int64_t(v.size()) > first && v.back().off + v.back().len <= off &&
          off - (v.back().off + v.back().len) <= gap)
        v.back().len = off + len - v.back().off;
      else
        v.push_back(CopyRange{off, len});
    };
    hp.layer_units.assign(1, 0);
    hp.payload_layer.assign(1, 0);
    hp.scale_layer.assign(1, 0);
    // Staged restore: per request, the reused blocks' K + V tile ranges
    // relative to a layer's payload start, in payload order.
    std::vector<std::vector<CopyRange>> reused(static_cast<size_t>(num_requests));
    std::vector<bool> scales_needed(static_cast<size_t>(num_requests), false);
    hp.stage_ok = true;
    for (int32_t r = 0; r < num_requests; ++r) {
      const pkv_request_t& q = requests[r];
      const int64_t nb = ceil_div(q.suffix_tokens, B);
      for (int tag = 0; tag < 4; ++tag)
        for (int64_t b = 0; b < nb; ++b)
          if (q.tags[b] == tag && !q.repair_mask[b]) {
            reused[size_t(r)].push_back(
                CopyRange{block_off[r][b], tile_bytes(m, kKeyBits[tag]) + tile_bytes(m, kValueBits[tag])});
            if (tag != PKV_TAG_FP16) scales_needed[size_t(r)] = true;
          }
      if (scales_needed[size_t(r)] && uint64_t(nb) * H * 4 * 2 > kStageScaleBytes) hp.stage_ok = false;
    }
    for (int64_t l = 0; l < L; ++l) {
      for (int32_t r = 0; r < num_requests; ++r) {
        const int64_t u_begin = int64_t(hp.units.size());
        const pkv_request_t& q = requests[r];
        const int64_t nb = ceil_div(q.suffix_tokens, B);
        const ReqInfo& rd = hp.reqs[r];
        const uint64_t layer_base = q.payload_offset + uint64_t(l) * layer_bytes[r];
        bool any_quantized = false;
        // Payload ranges in layout order (runs by tag, ascending blocks) so
        // that neighbouring reused blocks merge into one copy; merging stays
        // inside this request's layer, so copies never overlap.
        const int64_t first_range = int64_t(hp.payload_ranges.size());
        for (int tag = 0; tag < 4; ++tag)
          for (int64_t b = 0; b < nb; ++b)
            if (q.tags[b] == tag && !q.repair_mask[b]) {
              add_range(hp.payload_ranges, first_range, layer_base + block_off[r][b],
                        tile_bytes(m, kKeyBits[tag]) + tile_bytes(m, kValueBits[tag]), kHostGapBytes);
              any_quantized |= tag != PKV_TAG_FP16;
            }
        if (any_quantized)
          add_range(hp.scale_ranges, hp.scale_layer.back(), (q.scale_offset + uint64_t(l) * nb * H * 4) * 2,
                    uint64_t(nb) * H * 4 * 2, 0);
        for (int64_t b = 0; b < nb; ++b) {
          if (q.repair_mask[b]) continue;
          const int tag = q.tags[b];
          const int64_t n_valid = std::min<int64_t>(B, q.suffix_tokens - b * B);
          // Split the block into units of at most `per_unit` tokens that
          // never cross a page boundary, so a unit writes slots of one page.
          // A page's run of rows is cut into equal parts (17 -> 9 + 8, not 16 + 1).
          for (int64_t t0 = 0, len = 0; t0 < n_valid; t0 += len) {
            const int64_t run = std::min<int64_t>(P - ((q.dst_row0 + b * B + t0) & (P - 1)), n_valid - t0);
            len = ceil_div(run, ceil_div(run, per_unit));
            Unit u;
            const uint64_t block_base = layer_base + block_off[r][b];
            u.k_off = block_base + uint64_t(t0) * H * D * kKeyBits[tag] / 8;
            u.v_off = block_base + tile_bytes(m, kKeyBits[tag]) + uint64_t(t0) * H * D * kValueBits[tag] / 8;
            u.scale_off = q.scale_offset + (uint64_t(l) * nb + b) * H * 4;
            u.row0 = q.dst_row0 + b * B + t0;
            u.pt_off = rd.pt_off;
            u.table_off = int32_t(rd.table_off);
            u.layer = int32_t(l);
            u.tag = tag | (q.delta != 0 ? kUnitRotate : 0);
            u.n_valid = int32_t(len);
            u.page1 = q.page_table[(q.dst_row0 + b * B + t0) >> lp2];  // validated above; one page per unit
            u.page2 = 0;
            hp.units.push_back(u);
          }
          hp.info.restored_rows += n_valid;
          if (q.delta != 0) hp.rotated_rows += n_valid;
          hp.info.bytes_read += uint64_t(n_valid) * H * D * (kKeyBits[tag] + kValueBits[tag]) / 8;
          if (tag != PKV_TAG_FP16) hp.info.bytes_read += uint64_t(H) * 4 * 2;
        }
        if (hp.stage_ok && int64_t(hp.units.size()) > u_begin)
          add_stage_steps(hp, reused[size_t(r)], u_begin, int64_t(hp.units.size()), layer_base,
                          scales_needed[size_t(r)] ? (q.scale_offset + uint64_t(l) * nb * H * 4) : 0,
                          scales_needed[size_t(r)] ? uint64_t(nb) * H * 4 : 0);
      }
      hp.layer_units.push_back(int64_t(hp.units.size()));
      hp.payload_layer.push_back(int64_t(hp.payload_ranges.size()));
      hp.scale_layer.push_back(int64_t(hp.scale_ranges.size()));
    }
    for (const CopyRange& c : hp.payload_ranges) hp.info.host_copy_bytes += c.len;
    for (const CopyRange& c : hp.scale_ranges) hp.info.host_copy_bytes += c.len;
    for (const auto* v : {&hp.payload_ranges, &hp.scale_ranges})
      for (const CopyRange& c : *v) hp.info.host_copies += int64_t((c.len + kHostChunkBytes - 1) / kHostChunkBytes);
  } catch (const std::bad_alloc&) {
    return PKV_ERR_OUT_OF_MEMORY;
  }
  if (hp.units.size() > size_t(std::numeric_limits<int32_t>::max())) return PKV_ERR_INVALID_ARGUMENT;
  hp.info.num_units = int64_t(hp.units.size());
  hp.info.bytes_written = uint64_t(hp.info.restored_rows) * H * D * 2 * 2;
  return PKV_OK;
}

int32_t gather_workgroup(const pkv_model_t& m) {
  return 64 * std::min<int32_t>(m.num_kv_heads, kGatherMaxWaves);
}

pkv_status_t build_checkpoint_plan(const pkv_model_t* model, const pkv_checkpoint_request_t* requests,
                                   int32_t num_requests, HostPlan* out) {
  pkv_status_t st = check_model(model);
  if (st != PKV_OK) return st;
  if (num_requests < 0 || (num_requests > 0 && !requests) || !out) return PKV_ERR_INVALID_ARGUMENT;
  const pkv_model_t& m = *model;
  const int64_t B = m.block_tokens, H = m.num_kv_heads, D = m.head_dim, P = m.page_size, L = m.num_layers;
  const int lp2 = ilog2(P);
  // Fields and tags.
  for (int32_t r = 0; r < num_requests; ++r) {
    const pkv_checkpoint_request_t& q = requests[r];
    if (q.reserved != 0 || q.reserved2 != 0) return PKV_ERR_INVALID_ARGUMENT;
    if (q.suffix_tokens < 0 || q.num_logical_pages < 0 || q.src_row0 < 0 || q.src_row0 > (int64_t(1) << 50))
      return PKV_ERR_INVALID_ARGUMENT;
    if (q.suffix_tokens > 0 && !q.tags) return PKV_ERR_INVALID_ARGUMENT;
    if (q.num_logical_pages > 0 && !q.page_table) return PKV_ERR_INVALID_ARGUMENT;
    if (q.payload_offset % 16 != 0 || q.scale_offset % 4 != 0) return PKV_ERR_INVALID_ARGUMENT;
    if (q.payload_offset > (uint64_t(1) << 56) || q.scale_offset > (uint64_t(1) << 56)) return PKV_ERR_INVALID_ARGUMENT;
    const int64_t nb = ceil_div(q.suffix_tokens, B);
    for (int64_t b = 0; b < nb; ++b)
      if (q.tags[b] > PKV_TAG_K4V4) return PKV_ERR_BAD_TAG;
  }
  // Every source row on a mapped, in-range page.
  for (int32_t r = 0; r < num_requests; ++r) {
    const pkv_checkpoint_request_t& q = requests[r];
    if (q.suffix_tokens == 0) continue;
    const int64_t first = q.src_row0 >> lp2, last = (q.src_row0 + q.suffix_tokens - 1) >> lp2;
    for (int64_t lp = first; lp <= last; ++lp) {
      if (lp >= q.num_logical_pages) return PKV_ERR_PAGE_OUT_OF_RANGE;
      const int32_t pp = q.page_table[lp];
      if (pp == -1) return PKV_ERR_PAGE_UNMAPPED;
      if (pp < -1 || pp >= m.pool_pages) return PKV_ERR_PAGE_OUT_OF_RANGE;
    }
  }
  // Output ranges of different requests must not overlap.
  std::vector<std::pair<uint64_t, uint64_t>> pr, sr;
  for (int32_t r = 0; r < num_requests; ++r) {
    const pkv_checkpoint_request_t& q = requests[r];
    const int64_t nb = ceil_div(q.suffix_tokens, B);
    if (nb == 0) continue;
    pr.emplace_back(q.payload_offset, q.payload_offset + uint64_t(L) * layer_payload_bytes(m, q.tags, nb));
    sr.emplace_back(q.scale_offset, q.scale_offset + uint64_t(L) * nb * H * 4);
  }
  for (auto* v : {&pr, &sr}) {
    std::sort(v->begin(), v->end());
    for (size_t i = 1; i < v->size(); ++i)
      if ((*v)[i].first < (*v)[i - 1].second) return PKV_ERR_INVALID_ARGUMENT;
  }

  HostPlan& hp = *out;
  hp.kind = 1;
  hp.workgroup = gather_workgroup(m);
  hp.model = m;
  hp.log2_page = lp2;
  hp.units.clear();
  hp.reqs.clear();
  hp.tables.clear();
  hp.page_tables.clear();
  memset(&hp.info, 0, sizeof(hp.info));
  hp.info.num_requests = num_requests;
  hp.info.kind = 1;
  hp.info.cache_bytes = cache_bytes(m);
  try {
    hp.req_payload_bytes.assign(size_t(num_requests), 0);
    for (int32_t r = 0; r < num_requests; ++r) {
      const pkv_checkpoint_request_t& q = requests[r];
      const int64_t nb = ceil_div(q.suffix_tokens, B);
      const int64_t pt_off = int64_t(hp.page_tables.size());
      hp.page_tables.insert(hp.page_tables.end(), q.page_table, q.page_table + q.num_logical_pages);
      if (nb == 0) continue;
      std::vector<uint64_t> block_off(nb);
      uint64_t pos = 0;
      for (int tag = 0; tag < 4; ++tag)
        for (int64_t b = 0; b < nb; ++b)
          if (q.tags[b] == tag) {
            block_off[b] = pos;
            pos += tile_bytes(m, kKeyBits[tag]) + tile_bytes(m, kValueBits[tag]);
          }
      const uint64_t layer_bytes = pos;
      hp.req_payload_bytes[r] = uint64_t(L) * layer_bytes;
      hp.info.payload_bytes = std::max<uint64_t>(hp.info.payload_bytes, q.payload_offset + uint64_t(L) * layer_bytes);
      hp.info.scale_bytes = std::max<uint64_t>(hp.info.scale_bytes, (q.scale_offset + uint64_t(L) * nb * H * 4) * 2);
      for (int64_t l = 0; l < L; ++l) {
        for (int64_t b = 0; b < nb; ++b) {
          const int tag = q.tags[b];
          Unit u;
          u.k_off = q.payload_offset + uint64_t(l) * layer_bytes + block_off[b];
          u.v_off = u.k_off + tile_bytes(m, kKeyBits[tag]);
          u.scale_off = q.scale_offset + (uint64_t(l) * nb + b) * H * 4;
          u.row0 = q.src_row0 + b * B;
          u.pt_off = pt_off;
          u.layer = int32_t(l);
          u.tag = tag;
          u.n_valid = int32_t(std::min<int64_t>(B, q.suffix_tokens - b * B));
          const int64_t first = u.row0 >> lp2, last = (u.row0 + u.n_valid - 1) >> lp2;
          u.page0 = q.page_table[first];
          u.page1 = first + 1 <= last ? q.page_table[first + 1] : -1;
          u.page2 = first + 2 <= last ? q.page_table[first + 2] : -1;
          hp.units.push_back(u);
        }
        hp.info.bytes_written += layer_bytes + uint64_t(nb) * H * 4 * 2;
      }
      hp.info.restored_rows += int64_t(L) * q.suffix_tokens;
    }
  } catch (const std::bad_alloc&) {
    return PKV_ERR_OUT_OF_MEMORY;
  }
  if (hp.units.size() > size_t(std::numeric_limits<int32_t>::max())) return PKV_ERR_INVALID_ARGUMENT;
  hp.info.num_units = int64_t(hp.units.size());
  hp.info.bytes_read = uint64_t(hp.info.restored_rows) * H * D * 2 * 2;
  return PKV_OK;
}

}  // namespace pkv

extern "C" {

pkv_status_t pkv_payload_size(const pkv_model_t* model, const pkv_request_t* request, uint64_t* payload_bytes,
                              uint64_t* scale_elems) {
  pkv_status_t st = pkv::check_model(model);
  if (st != PKV_OK) return st;
  if (!request || !payload_bytes || !scale_elems) return PKV_ERR_INVALID_ARGUMENT;
  if (request->suffix_tokens < 0) return PKV_ERR_INVALID_ARGUMENT;
  const int64_t nb = pkv::ceil_div(request->suffix_tokens, model->block_tokens);
  if (nb > 0 && !request->tags) return PKV_ERR_INVALID_ARGUMENT;
  if ((st = pkv::check_tags(*request, nb)) != PKV_OK) return st;
  *payload_bytes = uint64_t(model->num_layers) * pkv::layer_payload_bytes(*model, request->tags, nb);
  *scale_elems = uint64_t(model->num_layers) * uint64_t(nb) * model->num_kv_heads * 4;
  return PKV_OK;
}

// Internal test hook (not part of pkv.h): the host-built work list, so tests
// can check every address the kernel derives from it without a GPU.
pkv_status_t pkv_internal_host_units(const pkv_model_t* model, const pkv_request_t* requests, int32_t num_requests,
                                     void* units_out, int64_t capacity, int64_t* count) {
  if (!count) return PKV_ERR_INVALID_ARGUMENT;
  pkv::HostPlan hp;
  pkv_status_t st = pkv::build_host_plan(model, requests, num_requests, &hp);
  if (st != PKV_OK) return st;
  *count = int64_t(hp.units.size());
  if (units_out && capacity >= *count && *count > 0)
    memcpy(units_out, hp.units.data(), hp.units.size() * sizeof(pkv::Unit));
  return PKV_OK;
}

// Internal test hook (not part of pkv.h): threads per restore workgroup.
pkv_status_t pkv_internal_restore_workgroup(const pkv_model_t* model, int32_t* threads) {
  if (!model || !threads) return PKV_ERR_INVALID_ARGUMENT;
  *threads = pkv::restore_workgroup(*model);
  return PKV_OK;
}

pkv_status_t pkv_plan_repair(int32_t suffix_tokens, int32_t block_tokens, int64_t dirty_tokens,
                             const float* importance, double kappa, uint8_t* repair_mask, int64_t* nonlocal_tokens) {
  if (suffix_tokens < 0 || block_tokens < 1 || block_tokens > pkv::kMaxBlockTokens || dirty_tokens < 0)
    return PKV_ERR_INVALID_ARGUMENT;
  if (!(kappa >= 0.0 && kappa <= 1.0)) return PKV_ERR_INVALID_ARGUMENT;
  const int64_t N = suffix_tokens, B = block_tokens, nb = (N + B - 1) / B;
  if (N > 0 && (!importance || !repair_mask)) return PKV_ERR_INVALID_ARGUMENT;
  for (int64_t i = 0; i < N; ++i)
    if (!std::isfinite(importance[i])) return PKV_ERR_INVALID_ARGUMENT;
  const int64_t d = std::min<int64_t>(dirty_tokens, N);
  const int64_t candidates = N - d;
  int64_t k = int64_t(std::floor(kappa * double(candidates) + 0.5));
  k = std::min<int64_t>(std::max<int64_t>(k, 0), candidates);
  try {
    std::vector<uint8_t> mask(size_t(nb), 0);
    // Eq. 9: the dirty window D = [0, d) rounds to blocks [0, ceil(d / B)).
    for (int64_t b = 0; b < (d + B - 1) / B; ++b) mask[size_t(b)] = 1;
    // Eq. 11: the k best-scoring candidates (score descending, index ascending).
    if (k > 0) {
      std::vector<std::pair<float, int32_t>> cand(static_cast<size_t>(candidates));
      for (int64_t i = 0; i < candidates; ++i) cand[size_t(i)] = {importance[d + i], int32_t(d + i)};
      auto better = [](const std::pair<float, int32_t>& a, const std::pair<float, int32_t>& b) {
        return a.first > b.first || (a.first == b.first && a.second < b.second);
      };
      if (k < candidates) std::nth_element(cand.begin(), cand.begin() + (k - 1), cand.end(), better);
      for (int64_t j = 0; j < k; ++j) mask[size_t(cand[size_t(j)].second / B)] = 1;  // Eq. 12
    }
    std::copy(mask.begin(), mask.end(), repair_mask);
  } catch (const std::bad_alloc&) {
    return PKV_ERR_OUT_OF_MEMORY;
  }
  if (nonlocal_tokens) *nonlocal_tokens = k;
  return PKV_OK;
}

// Internal test hook (not part of pkv.h): the (cos, sin) tables of a restore
// plan, [num_requests][D/2][2] in the kernel's element order.
pkv_status_t pkv_internal_host_tables(const pkv_model_t* model, const pkv_request_t* requests, int32_t num_requests,
                                      double* out, int64_t capacity, int64_t* count) {
  if (!count) return PKV_ERR_INVALID_ARGUMENT;
  pkv::HostPlan hp;
  pkv_status_t st = pkv::build_host_plan(model, requests, num_requests, &hp);
  if (st != PKV_OK) return st;
  *count = int64_t(hp.tables.size());
  if (out && capacity >= *count && *count > 0) memcpy(out, hp.tables.data(), hp.tables.size() * sizeof(double));
  return PKV_OK;
}

// Internal test hook (not part of pkv.h): the gap below which the streamed
// restore merges two copies of one layer.
uint64_t pkv_internal_host_gap_bytes() { return pkv::kHostGapBytes; }

// Internal test hook (not part of pkv.h): the streamed restore's schedule.
// ranges_out receives (offset, length) byte pairs, payload ranges first,
// then scale ranges; layers_out receives [3][L + 1] starts: units, payload
// ranges, scale ranges.  Counts are returned even when the buffers are short.
pkv_status_t pkv_internal_stream_schedule(const pkv_model_t* model, const pkv_request_t* requests,
                                          int32_t num_requests, uint64_t* ranges_out, int64_t capacity,
                                          int64_t* n_payload, int64_t* n_scale, int64_t* layers_out) {
  if (!n_payload || !n_scale || !layers_out || !model) return PKV_ERR_INVALID_ARGUMENT;
  pkv::HostPlan hp;
  pkv_status_t st = pkv::build_host_plan(model, requests, num_requests, &hp);
  if (st != PKV_OK) return st;
  *n_payload = int64_t(hp.payload_ranges.size());
  *n_scale = int64_t(hp.scale_ranges.size());
  const size_t L1 = size_t(model->num_layers) + 1;
  for (size_t i = 0; i < L1; ++i) {
    layers_out[i] = hp.layer_units[i];
    layers_out[L1 + i] = hp.payload_layer[i];
    layers_out[2 * L1 + i] = hp.scale_layer[i];
  }
  if (ranges_out && capacity >= *n_payload + *n_scale) {
    size_t k = 0;
    for (const auto* v : {&hp.payload_ranges, &hp.scale_ranges})
      for (const pkv::CopyRange& c : *v) {
        ranges_out[2 * k] = c.off;
        ranges_out[2 * k + 1] = c.len;
        ++k;
      }
  }
  return PKV_OK;
}

// Internal test hook (not part of pkv.h): the schedule of the staged
// (allocation-free) restore.  steps_out receives 8 int64 per step (u0, u1,
// win_lo, win_hi, scale0, scale_elems, copy0, copy1), copies_out 3 uint64 per
// copy (src, dst, len); *stage_ok is 0 when the plan cannot be staged.
// Counts are returned even when the buffers are short.
pkv_status_t pkv_internal_stage_schedule(const pkv_model_t* model, const pkv_request_t* requests,
                                         int32_t num_requests, int64_t* steps_out, int64_t step_capacity,
                                         uint64_t* copies_out, int64_t copy_capacity, int64_t* n_steps,
                                         int64_t* n_copies, int32_t* stage_ok) {
  if (!n_steps || !n_copies || !stage_ok) return PKV_ERR_INVALID_ARGUMENT;
  pkv::HostPlan hp;
  pkv_status_t st = pkv::build_host_plan(model, requests, num_requests, &hp);
  if (st != PKV_OK) return st;
  *n_steps = int64_t(hp.stage_steps.size());
  *n_copies = int64_t(hp.stage_copies.size());
  *stage_ok = hp.stage_ok ? 1 : 0;
  if (steps_out && step_capacity >= *n_steps)
    for (size_t i = 0; i < hp.stage_steps.size(); ++i) {
      const pkv::StageStep& s = hp.stage_steps[i];
      const int64_t v[8] = {s.u0, s.u1, int64_t(s.win_lo), int64_t(s.win_hi), int64_t(s.scale0),
                            int64_t(s.scale_elems), s.copy0, s.copy1};
      memcpy(steps_out + 8 * i, v, sizeof(v));
    }
  if (copies_out && copy_capacity >= *n_copies)
    for (size_t i = 0; i < hp.stage_copies.size(); ++i) {
      copies_out[3 * i] = hp.stage_copies[i].src;
      copies_out[3 * i + 1] = hp.stage_copies[i].dst;
      copies_out[3 * i + 2] = hp.stage_copies[i].len;
    }
  return PKV_OK;
}

// Internal test hook (not part of pkv.h): the work list of a checkpoint plan.
pkv_status_t pkv_internal_checkpoint_units(const pkv_model_t* model, const pkv_checkpoint_request_t* requests,
                                           int32_t num_requests, void* units_out, int64_t capacity, int64_t* count,
                                           int32_t* workgroup) {
  if (!count || !workgroup) return PKV_ERR_INVALID_ARGUMENT;
  pkv::HostPlan hp;
  pkv_status_t st = pkv::build_checkpoint_plan(model, requests, num_requests, &hp);
  if (st != PKV_OK) return st;
  *count = int64_t(hp.units.size());
  *workgroup = hp.workgroup;
  if (units_out && capacity >= *count && *count > 0)
    memcpy(units_out, hp.units.data(), hp.units.size() * sizeof(pkv::Unit));
  return PKV_OK;
}

const char* pkv_status_string(pkv_status_t s) {
  switch (s) {
    case PKV_OK: return "ok";
    case PKV_ERR_INVALID_ARGUMENT: return "invalid argument";
    case PKV_ERR_BAD_TAG: return "bad precision tag";
    case PKV_ERR_PAGE_OUT_OF_RANGE: return "page out of range";
    case PKV_ERR_PAGE_UNMAPPED: return "page unmapped";
    case PKV_ERR_PAGE_ALIAS: return "physical page written through two logical pages";
    case PKV_ERR_OUT_OF_MEMORY: return "out of memory";
    case PKV_ERR_DEVICE: return "device error";
  }
  return "unknown status";
}

}  // extern "C"
