// Checkpoint write (PatchKV Section IV-D, offload side): gather a block's
// rows from the old context's paged cache, compute per-(block, head, K|V)
// binary16 scale and zero, pack FP16 / 8-bit / 4-bit codes and place them in
// the clustered checkpoint layout that the restore kernel reads.
//
// One workgroup encodes one (request, layer, block): every head, every row
// (padding rows of a partial last block are written as code 0 / +0).  A
// thread owns the same piece as in the restore kernel -- channels [8j, 8j+8)
// and [D/2+8j, D/2+8j+8) of one head -- for up to 4 tokens, and keeps the
// block's values in registers between the min/max pass and the encode pass,
// so the cache is read once.  The per-head min and max are combined with LDS
// integer atomics on order-preserving keys of the float values.
//
// Arithmetic follows the format's definition exactly: the zero is the
// largest binary16 not above the minimum, the scale the smallest binary16
// not below (max - zero)/(2^bits - 1) (both computed in double), and a code
// is round-half-even((x - zero)/scale).  The quotient is formed as
// (x - zero) * (1/scale) in double and, whenever that lands within 1e-6 of a
// rounding boundary, recomputed with a true division, so the codes equal those
// of a correctly rounded division.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <new>

#include "pkv.h"
#include "pkv_internal.h"

namespace pkv {
namespace {

struct GatherArgs {
  const Unit* units;
  const int32_t* page_tables;
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  uint8_t* payload;
  uint16_t* scales;
  int64_t layer_elems;
  int32_t H, D, B, log2P, cols, tpp;
};

__device__ __forceinline__ int32_t order_key(float f) {
  const int32_t b = __float_as_int(f);
  return b ^ ((b >> 31) & 0x7FFFFFFF);
}
__device__ __forceinline__ float from_order_key(int32_t k) { return __int_as_float(k ^ ((k >> 31) & 0x7FFFFFFF)); }

template <bool BF16>
__device__ __forceinline__ float cache_value(uint32_t bits16) {
  if constexpr (BF16) {
    return __uint_as_float(bits16 << 16);
  } else {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(bits16)));
  }
}

// binary16 helpers.  The double -> binary16 cast is a single correctly
// rounded conversion (round to nearest even).
__device__ __forceinline__ uint16_t f16_nearest(double d) {
  return __builtin_bit_cast(uint16_t, static_cast<_Float16>(d));
}
__device__ __forceinline__ double f16_value(uint16_t b) {
  return static_cast<double>(static_cast<float>(__builtin_bit_cast(_Float16, b)));
}
__device__ __forceinline__ uint16_t f16_next_down(uint16_t b) {
  if (b & 0x8000) return uint16_t(b + 1);
  return (b & 0x7FFF) == 0 ? uint16_t(0x8001) : uint16_t(b - 1);
}
__device__ __forceinline__ uint16_t f16_next_up(uint16_t b) {
  if (!(b & 0x8000)) return uint16_t(b + 1);
  return (b & 0x7FFF) == 0 ? uint16_t(0x0001) : uint16_t(b - 1);
}
__device__ __forceinline__ uint16_t f16_floor(double x) {
  const uint16_t h = f16_nearest(x);
  return f16_value(h) > x ? f16_next_down(h) : h;
}
__device__ __forceinline__ uint16_t f16_ceil(double x) {
  const uint16_t h = f16_nearest(x);
  return f16_value(h) < x ? f16_next_up(h) : h;
}

__device__ __forceinline__ uint32_t element(const uint4& w, int e) {
  const uint32_t word = e < 2 ? w.x : e < 4 ? w.y : e < 6 ? w.z : w.w;
  return (word >> (16 * (e & 1))) & 0xFFFFu;
}

// Code of one value: round-half-even((x - zero) / scale), clipped.
__device__ __forceinline__ uint32_t encode(float x, double zero, double scale, double inv, double qmax) {
  if (scale == 0.0) return 0;
  const double d = static_cast<double>(x) - zero;  // exact
  const double y = d * inv;
  double k = __builtin_rint(y);
  if (__builtin_fabs(__builtin_fabs(y - k) - 0.5) < 1e-6) k = __builtin_rint(d / scale);
  k = k < 0.0 ? 0.0 : (k > qmax ? qmax : k);
  return static_cast<uint32_t>(k);
}

template <bool BF16>
__device__ __forceinline__ uint4 to_half8(const uint4& w) {
  if constexpr (!BF16) {
    return w;
  } else {
    uint32_t o[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const uint16_t lo = __builtin_bit_cast(uint16_t, static_cast<_Float16>(cache_value<true>(element(w, 2 * p))));
      const uint16_t hi = __builtin_bit_cast(uint16_t, static_cast<_Float16>(cache_value<true>(element(w, 2 * p + 1))));
      o[p] = uint32_t(lo) | (uint32_t(hi) << 16);
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// Encode one K or V tile of the unit's block (all rows) and its scales.
template <bool BF16>
__device__ void encode_tile(const GatherArgs& a, const Unit& u, const uint16_t* __restrict__ cache,
                            uint8_t* __restrict__ tile, int which, int bits, int32_t* s_min, int32_t* s_max,
                            bool active, int t0, int head, int j) {
  const int H = a.H, D = a.D;
  const int64_t slot_mask = (int64_t(1) << a.log2P) - 1;
  const int64_t row_elems = int64_t(H) * D;
  const int64_t lbase = int64_t(u.layer) * a.layer_elems + int64_t(head) * D;
  uint4 lo[kGatherTokens], hi[kGatherTokens];
#pragma unroll
  for (int i = 0; i < kGatherTokens; ++i) {
    lo[i] = make_uint4(0, 0, 0, 0);
    hi[i] = make_uint4(0, 0, 0, 0);
    const int t = t0 + i * a.tpp;
    if (active && t < u.n_valid) {
      const int64_t row = u.row0 + t;
      const int64_t page = a.page_tables[u.pt_off + (row >> a.log2P)];
      const uint16_t* src = cache + lbase + ((page << a.log2P) | (row & slot_mask)) * row_elems;
      lo[i] = *reinterpret_cast<const uint4*>(src + 8 * j);
      hi[i] = *reinterpret_cast<const uint4*>(src + D / 2 + 8 * j);
    }
  }
  const bool scale_writer = active && t0 == 0 && j == 0;
  if (bits == 16) {
#pragma unroll
    for (int i = 0; i < kGatherTokens; ++i) {
      const int t = t0 + i * a.tpp;
      if (active && t < a.B) {
        uint8_t* row = tile + (int64_t(t) * H + head) * D * 2;
        *reinterpret_cast<uint4*>(row + 16 * j) = to_half8<BF16>(lo[i]);
        *reinterpret_cast<uint4*>(row + D + 16 * j) = to_half8<BF16>(hi[i]);
      }
    }
    if (scale_writer) {
      *reinterpret_cast<uint32_t*>(a.scales + u.scale_off + 4 * head + 2 * which) = 0u;
    }
    return;
  }
  // Per-head range over the valid rows.
  float mn = __builtin_inff(), mx = -__builtin_inff();
#pragma unroll
  for (int i = 0; i < kGatherTokens; ++i) {
    const int t = t0 + i * a.tpp;
    if (active && t < u.n_valid) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x0 = cache_value<BF16>(element(lo[i], e));
        const float x1 = cache_value<BF16>(element(hi[i], e));
        mn = __builtin_fminf(mn, __builtin_fminf(x0, x1));
        mx = __builtin_fmaxf(mx, __builtin_fmaxf(x0, x1));
      }
    }
  }
  if (active) {
    atomicMin(&s_min[head], order_key(mn));
    atomicMax(&s_max[head], order_key(mx));
  }
  __syncthreads();
  const double qmax = double((1 << bits) - 1);
  const double vmin = static_cast<double>(from_order_key(s_min[head])) + 0.0;  // -0 counts as +0
  const double vmax = static_cast<double>(from_order_key(s_max[head]));
  const uint16_t zb = f16_floor(vmin);
  const double zero = f16_value(zb);
  const uint16_t sb = f16_ceil(((vmax - zero) + 0.0) / qmax);  // -0 span counts as +0
  const double scale = f16_value(sb);
  const double inv = scale != 0.0 ? 1.0 / scale : 0.0;
#pragma unroll
  for (int i = 0; i < kGatherTokens; ++i) {
    const int t = t0 + i * a.tpp;
    if (!(active && t < a.B)) continue;
    uint32_t c[16];
    const bool valid = t < u.n_valid;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      c[e] = valid ? encode(cache_value<BF16>(element(lo[i], e)), zero, scale, inv, qmax) : 0u;
      c[8 + e] = valid ? encode(cache_value<BF16>(element(hi[i], e)), zero, scale, inv, qmax) : 0u;
    }
    const int64_t r = int64_t(t) * H + head;
    if (bits == 8) {
      uint8_t* row = tile + r * D;
      const uint2 w0 = make_uint2(c[0] | (c[1] << 8) | (c[2] << 16) | (c[3] << 24),
                                  c[4] | (c[5] << 8) | (c[6] << 16) | (c[7] << 24));
      const uint2 w1 = make_uint2(c[8] | (c[9] << 8) | (c[10] << 16) | (c[11] << 24),
                                  c[12] | (c[13] << 8) | (c[14] << 16) | (c[15] << 24));
      *reinterpret_cast<uint2*>(row + 8 * j) = w0;
      *reinterpret_cast<uint2*>(row + D / 2 + 8 * j) = w1;
    } else {
      uint8_t* row = tile + r * (D / 2);
      uint32_t w0 = 0, w1 = 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        w0 |= c[e] << (4 * e);
        w1 |= c[8 + e] << (4 * e);
      }
      *reinterpret_cast<uint32_t*>(row + 4 * j) = w0;
      *reinterpret_cast<uint32_t*>(row + D / 4 + 4 * j) = w1;
    }
  }
  if (scale_writer) {
    *reinterpret_cast<uint32_t*>(a.scales + u.scale_off + 4 * head + 2 * which) = uint32_t(sb) | (uint32_t(zb) << 16);
  }
}

template <bool BF16>
__global__ __launch_bounds__(1024) void gather_kernel(GatherArgs a) {
  __shared__ int32_t s_min[kMaxRowElems / 16];
  __shared__ int32_t s_max[kMaxRowElems / 16];
  const Unit u = a.units[blockIdx.x];
  const int tid = threadIdx.x;
  const int tag = u.tag & 0xFF;
  const int t0 = tid / a.cols;
  const bool active = t0 < a.tpp;
  const int c = tid - t0 * a.cols;
  const int dq = a.D >> 4;
  const int head = active ? c / dq : 0;
  const int j = active ? c - head * dq : 0;
  for (int which = 0; which < 2; ++which) {
    const int bits = which == 0 ? kKeyBits[tag] : kValueBits[tag];
    if (bits != 16) {
      for (int h = tid; h < a.H; h += blockDim.x) {
        s_min[h] = order_key(__builtin_inff());
        s_max[h] = order_key(-__builtin_inff());
      }
      __syncthreads();
    }
    encode_tile<BF16>(a, u, which == 0 ? a.k_cache : a.v_cache, a.payload + (which == 0 ? u.k_off : u.v_off), which,
                      bits, s_min, s_max, active, t0, head, j);
    __syncthreads();  // the next tile reuses the LDS range
  }
}

bool overlap(const void* a, uint64_t na, const void* b, uint64_t nb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}

}  // namespace
}  // namespace pkv

extern "C" {

pkv_status_t pkv_checkpoint_plan(const pkv_model_t* model, const pkv_checkpoint_request_t* requests,
                                 int32_t num_requests, pkv_plan_t** out) {
  if (!out) return PKV_ERR_INVALID_ARGUMENT;
  *out = nullptr;
  pkv::HostPlan hp;
  const pkv_status_t st = pkv::build_checkpoint_plan(model, requests, num_requests, &hp);
  if (st != PKV_OK) return st;
  return pkv::upload_plan(std::move(hp), out);
}

pkv_status_t pkv_quantize_gather(const pkv_plan_t* plan, const void* k_cache, const void* v_cache,
                                 uint64_t cache_bytes, void* payload, uint64_t payload_bytes, void* scales,
                                 uint64_t scale_bytes, void* hip_stream) {
  if (!plan || plan->host.kind != 1) return PKV_ERR_INVALID_ARGUMENT;
  const pkv_plan_info_t& info = plan->host.info;
  if (info.num_units == 0) return PKV_OK;
  if (!payload || !scales || !k_cache || !v_cache) return PKV_ERR_INVALID_ARGUMENT;
  if (reinterpret_cast<uintptr_t>(payload) % 16 || reinterpret_cast<uintptr_t>(scales) % 8 ||
      reinterpret_cast<uintptr_t>(k_cache) % 16 || reinterpret_cast<uintptr_t>(v_cache) % 16)
    return PKV_ERR_INVALID_ARGUMENT;
  if (payload_bytes < info.payload_bytes || scale_bytes < info.scale_bytes || cache_bytes < info.cache_bytes)
    return PKV_ERR_INVALID_ARGUMENT;
  const uint64_t cb = info.cache_bytes, pb = info.payload_bytes, sb = info.scale_bytes;
  if (pkv::overlap(payload, pb, scales, sb) || pkv::overlap(payload, pb, k_cache, cb) ||
      pkv::overlap(payload, pb, v_cache, cb) || pkv::overlap(scales, sb, k_cache, cb) ||
      pkv::overlap(scales, sb, v_cache, cb))
    return PKV_ERR_INVALID_ARGUMENT;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != plan->device) return PKV_ERR_DEVICE;

  const pkv_model_t& m = plan->host.model;
  pkv::GatherArgs a;
  a.units = plan->d_units;
  a.page_tables = plan->d_page_tables;
  a.k_cache = static_cast<const uint16_t*>(k_cache);
  a.v_cache = static_cast<const uint16_t*>(v_cache);
  a.payload = static_cast<uint8_t*>(payload);
  a.scales = static_cast<uint16_t*>(scales);
  a.layer_elems = m.pool_pages * int64_t(m.page_size) * m.num_kv_heads * m.head_dim;
  a.H = m.num_kv_heads;
  a.D = m.head_dim;
  a.B = m.block_tokens;
  a.log2P = plan->host.log2_page;
  a.cols = m.num_kv_heads * m.head_dim / 16;
  a.tpp = plan->host.workgroup / a.cols;
  const dim3 grid(static_cast<uint32_t>(info.num_units)), block(plan->host.workgroup);
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  if (m.out_dtype == PKV_OUT_BF16)
    hipLaunchKernelGGL(pkv::gather_kernel<true>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(pkv::gather_kernel<false>, grid, block, 0, stream, a);
  return hipGetLastError() == hipSuccess ? PKV_OK : PKV_ERR_DEVICE;
}

}  // extern "C"
