// Checkpoint write (PatchKV Section IV-D, offload side): gather a block's
// rows from the old context's paged cache, compute per-(block, head, K|V)
// binary16 scale and zero, pack FP16 / 8-bit / 4-bit codes and place them in
// the clustered checkpoint layout that the restore kernel reads.
//
// Work is split into tiles, one per (request, layer, block, K|V, head); one
// wave encodes one tile.  A wave's lanes cover a head's row in pieces of 8
// channels (D/8 lanes per row, 64/(D/8) rows per load), so the tile's
// min/max is a wave reduction: no LDS and no barrier.  A lane holds its rows
// in NL 16-byte registers between the range pass and the encode pass.
//
// Three kernels.  The tile kernel (blocks whose tile fits NL <= 8 loads per
// lane and spans at most three cache pages, layer slices below 4 GiB; tiles
// of 9 to 16 loads go to its two-waves-per-tile form) takes the
// block's source pages from its work item, so no page-table load sits in
// front of the row loads; it uses 32-bit buffer offsets, consumes every
// loaded register on every path, and issues every store (lanes with nothing
// to write get an offset the hardware drops), which keeps register use low
// and occupancy high.  The general kernel (any valid model) reads the page
// table per row and reads a tile twice when it needs more than 16 loads per
// lane (range pass, then encode pass).  In
// both, the waves of one workgroup encode the heads of one (block, K|V), so
// they write neighbouring pieces of the same rows into one L2.
//
// Arithmetic follows the format's definition exactly: the zero is the
// largest binary16 not above the minimum, the scale the smallest binary16
// not below (max - zero)/(2^bits - 1) (both in double), and a code is
// round-half-even((x - zero)/scale) with the quotient correctly rounded in
// double.  Codes are first formed in float: t = (x - zero) * (1/scale), which
// is within 5e-5 of the exact quotient (three roundings of 2^-24 relative on
// a quotient <= 255), rounded to the nearest integer by the hardware's float
// to byte conversion.  Whenever t lies farther than 1e-4 from a half-integer
// that is the exact rounding, and it never exceeds 2^bits - 1 (the scale is
// rounded up), so no clip is needed; a packed word of codes (8 four-bit or 4
// eight-bit) with any t closer to a half-integer is recomputed in double with
// a true division.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <new>

#include "pkv.h"
#include "pkv_internal.h"

namespace pkv {
namespace {

#ifndef GATHER_MIN_WAVES
#define GATHER_MIN_WAVES 1
#endif

struct GatherArgs {
  const Unit* units;
  const int32_t* page_tables;
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  uint8_t* payload;
  uint16_t* scales;
  int64_t layer_elems;  // elements of one layer of a cache (twice pool_pages * P * H * D when paired)
  int32_t H, D, B, log2P;
  int32_t page_shift;    // slot rows from a layer's start to page p: p << page_shift
  int32_t lpr;     // lanes per row: D / 8
  int32_t rpl;     // rows per load: 64 / lpr
  int32_t nchunk;  // register-resident chunks of NL loads per lane covering the block
};

template <bool BF16>
__device__ __forceinline__ float cache_value(uint32_t word, int half) {
  if constexpr (BF16) {
    return __uint_as_float(half ? (word & 0xFFFF0000u) : (word << 16));
  } else {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(half ? word >> 16 : word)));
  }
}

__device__ __forceinline__ uint32_t word_of(const uint4& w, int e) {
  return e < 2 ? w.x : e < 4 ? w.y : e < 6 ? w.z : w.w;
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

struct Quant {
  float zf, invf;
  uint32_t qmax;
  double zero, scale;
};

// Codes of the first N values of w (zero <= x <= max of the tile) packed into
// one word: N = 8 four-bit codes (nibble e) or N = 4 eight-bit codes (byte e).
// t = (x - zero) * (1/scale) is formed in float and v_cvt_pk_u8_f32 rounds it
// to nearest even into a byte (it saturates to [0, 255]; t never leaves
// [0, 2^bits - 1] by more than 5e-5, so no code needs a clip).  Four-bit codes
// of even and odd channels go to the bytes of two words that are then merged
// nibble-wise.  `near` is set when some t lies within 1e-4 of a half-integer,
// where the float quotient cannot decide the rounding; the caller then uses
// encode_exact.  With scale 0 (invf = 0) every t is 0.
constexpr float kTieWindow = 1e-4f;

template <bool BF16, int N>
__device__ __forceinline__ uint32_t encode_fast(const uint4& w, const Quant& q, bool& near) {
  uint32_t lo = 0, hi = 0;  // N == 4: the codes; N == 8: even / odd channels, one per byte
  float dist = 1.0f;        // min over values of |frac(t) - 1/2|
#pragma unroll
  for (int e = 0; e < N; ++e) {
    const float x = cache_value<BF16>(word_of(w, e), e & 1);
    const float t = (x - q.zf) * q.invf;
    if (N == 4 || !(e & 1))
      lo = __builtin_amdgcn_cvt_pk_u8_f32(t, N == 4 ? e : e >> 1, lo);
    else
      hi = __builtin_amdgcn_cvt_pk_u8_f32(t, e >> 1, hi);
    dist = __builtin_fminf(dist, __builtin_fabsf(__builtin_amdgcn_fractf(t) - 0.5f));
  }
  near = dist < kTieWindow;
  return N == 4 ? lo : lo | (hi << 4);
}

// The same codes from the definition in double: rint((x - zero) / scale)
// with a correctly rounded division, clipped.
template <bool BF16, int N>
__device__ __forceinline__ uint32_t encode_exact(uint4 w, const Quant& q) {
  constexpr int kBits = 32 / N;
  uint32_t packed = 0;
  for (int e = 0; e < N; ++e) {
    const uint32_t word = e < 2 ? w.x : e < 4 ? w.y : e < 6 ? w.z : w.w;
    const float x = cache_value<BF16>(word, e & 1);
    double k = __builtin_rint((static_cast<double>(x) - q.zero) / q.scale);
    k = k < 0.0 ? 0.0 : k;
    const uint32_t c = static_cast<uint32_t>(k);
    packed |= (c < q.qmax ? c : q.qmax) << (kBits * e);
  }
  return packed;
}

template <bool BF16, int N>
__device__ __forceinline__ uint32_t encode_word(const uint4& w, const Quant& q) {
  bool near;
  const uint32_t packed = encode_fast<BF16, N>(w, q, near);
  return near ? encode_exact<BF16, N>(w, q) : packed;
}

template <bool BF16>
__device__ __forceinline__ uint4 to_half8(const uint4& w) {
  if constexpr (!BF16) {
    return w;
  } else {
    uint32_t o[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const uint32_t word = word_of(w, 2 * p);
      const uint16_t lo = __builtin_bit_cast(uint16_t, static_cast<_Float16>(cache_value<true>(word, 0)));
      const uint16_t hi = __builtin_bit_cast(uint16_t, static_cast<_Float16>(cache_value<true>(word, 1)));
      o[p] = uint32_t(lo) | (uint32_t(hi) << 16);
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// Lane-private view of one (block, head, K|V) tile.
struct TileLane {
  const uint16_t* src;  // cache + layer + head + lane's channel piece
  uint8_t* tile;        // the tile's first byte
  int64_t row0, pt_off, row_elems, slot_mask;
  int32_t r, c, n_valid, log2P;
  bool on;              // lane holds a piece of a row
};

template <int NL>
__device__ __forceinline__ void load_chunk(const GatherArgs& a, const TileLane& L, int ch, uint4 (&w)[NL]) {
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int t = (ch * NL + i) * a.rpl + L.r;
    w[i] = make_uint4(0, 0, 0, 0);
    if (L.on && t < L.n_valid) {
      const int64_t row = L.row0 + t;
      const int64_t page = a.page_tables[L.pt_off + (row >> L.log2P)];
      w[i] = *reinterpret_cast<const uint4*>(L.src + ((page << a.page_shift) | (row & L.slot_mask)) * L.row_elems);
    }
  }
}

template <bool BF16, int NL>
__device__ void encode_tile(const GatherArgs& a, const Unit& u, int which, int head, int r, int c, bool on) {
  const int tag = u.tag & 0xFF;
  const int bits = which ? kValueBits[tag] : kKeyBits[tag];
  const int H = a.H, D = a.D;
  TileLane L;
  L.src = (which ? a.v_cache : a.k_cache) + int64_t(u.layer) * a.layer_elems + int64_t(head) * D + 8 * c;
  L.tile = a.payload + (which ? u.v_off : u.k_off);
  L.row0 = u.row0;
  L.pt_off = u.pt_off;
  L.row_elems = int64_t(H) * D;
  L.slot_mask = (int64_t(1) << a.log2P) - 1;
  L.r = r;
  L.c = c;
  L.n_valid = u.n_valid;
  L.log2P = a.log2P;
  L.on = on;
  uint32_t* scale_word = reinterpret_cast<uint32_t*>(a.scales + u.scale_off + 4 * head + 2 * which);
  const bool lane0 = (threadIdx.x & 63) == 0;
  uint4 w[NL];

  if (bits == 16) {
    for (int ch = 0; ch < a.nchunk; ++ch) {
      load_chunk<NL>(a, L, ch, w);
#pragma unroll
      for (int i = 0; i < NL; ++i) {
        const int t = (ch * NL + i) * a.rpl + r;
        if (on && t < a.B)
          *reinterpret_cast<uint4*>(L.tile + (int64_t(t) * H + head) * D * 2 + 16 * c) = to_half8<BF16>(w[i]);
      }
    }
    if (lane0) *scale_word = 0u;
    return;
  }

  // Range pass over the valid rows (padding rows load as 0 and are skipped).
  float mn = __builtin_inff(), mx = -__builtin_inff();
  for (int ch = 0; ch < a.nchunk; ++ch) {
    load_chunk<NL>(a, L, ch, w);
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int t = (ch * NL + i) * a.rpl + r;
      if (on && t < L.n_valid) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float x = cache_value<BF16>(word_of(w[i], e), e & 1);
          mn = __builtin_fminf(mn, x);
          mx = __builtin_fmaxf(mx, x);
        }
      }
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    mn = __builtin_fminf(mn, __shfl_xor(mn, off));
    mx = __builtin_fmaxf(mx, __shfl_xor(mx, off));
  }
  const double qmax = double((1 << bits) - 1);
  const double vmin = static_cast<double>(mn) + 0.0;  // -0 counts as +0
  const uint16_t zb = f16_floor(vmin);
  Quant q;
  q.zero = f16_value(zb);
  const uint16_t sb = f16_ceil(((static_cast<double>(mx) - q.zero) + 0.0) / qmax);  // -0 span counts as +0
  q.scale = f16_value(sb);
  q.zf = static_cast<float>(q.zero);
  q.invf = q.scale != 0.0 ? static_cast<float>(1.0 / q.scale) : 0.0f;
  q.qmax = uint32_t((1 << bits) - 1);
  const bool flat = q.scale == 0.0;  // every value equals the zero: code 0

  // Encode pass.
  for (int ch = 0; ch < a.nchunk; ++ch) {
    if (a.nchunk > 1) load_chunk<NL>(a, L, ch, w);
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int t = (ch * NL + i) * a.rpl + r;
      if (!(on && t < a.B)) continue;
      const bool valid = t < L.n_valid && !flat;
      if (bits == 8) {
        uint2 v = make_uint2(0, 0);
        if (valid) {
          v.x = encode_word<BF16, 4>(make_uint4(w[i].x, w[i].y, 0, 0), q);
          v.y = encode_word<BF16, 4>(make_uint4(w[i].z, w[i].w, 0, 0), q);
        }
        *reinterpret_cast<uint2*>(L.tile + (int64_t(t) * H + head) * D + 8 * c) = v;
      } else {
        const uint32_t v = valid ? encode_word<BF16, 8>(w[i], q) : 0u;
        *reinterpret_cast<uint32_t*>(L.tile + (int64_t(t) * H + head) * (D / 2) + 4 * c) = v;
      }
    }
  }
  if (lane0) *scale_word = uint32_t(sb) | (uint32_t(zb) << 16);
}

template <bool BF16, int NL>
__global__ __launch_bounds__(kGatherMaxWaves * 64, GATHER_MIN_WAVES) void gather_kernel(GatherArgs a) {
  const int64_t g = xcd_grouped(blockIdx.x, gridDim.x);
  const Unit u = a.units[g >> 1];
  const int which = int(g & 1);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nwaves = blockDim.x >> 6;
  const int r = lane / a.lpr;
  const int c = lane - r * a.lpr;
  const bool on = r < a.rpl;
  for (int head = wave; head < a.H; head += nwaves) encode_tile<BF16, NL>(a, u, which, head, r, c, on);
}

// ---------------------------------------------------------------------------
// Tile kernel for blocks that fit in registers (NL <= 8 loads per lane)
// and span at most three pages.  Workgroup b's wave w encodes tile
// b * waves + w of the (unit, K|V, head) order; the unit header, with the
// block's source pages, is one uniform scalar load; the tile's range is a DPP
// wave reduction (no LDS traffic, no barrier).
// ---------------------------------------------------------------------------

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_from(float identity, float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(identity), __float_as_int(v), CTRL, ROW_MASK, 0xF,
                                                    false));
}

// Min and max over the 64 lanes (every lane active), as uniform values.
__device__ __forceinline__ void wave_range(float& mn, float& mx) {
  const float pinf = __builtin_inff(), ninf = -__builtin_inff();
  mn = __builtin_fminf(mn, dpp_from<0x111, 0xF>(pinf, mn));  // row_shr:1
  mx = __builtin_fmaxf(mx, dpp_from<0x111, 0xF>(ninf, mx));
  mn = __builtin_fminf(mn, dpp_from<0x112, 0xF>(pinf, mn));  // row_shr:2
  mx = __builtin_fmaxf(mx, dpp_from<0x112, 0xF>(ninf, mx));
  mn = __builtin_fminf(mn, dpp_from<0x114, 0xF>(pinf, mn));  // row_shr:4
  mx = __builtin_fmaxf(mx, dpp_from<0x114, 0xF>(ninf, mx));
  mn = __builtin_fminf(mn, dpp_from<0x118, 0xF>(pinf, mn));  // row_shr:8
  mx = __builtin_fmaxf(mx, dpp_from<0x118, 0xF>(ninf, mx));
  mn = __builtin_fminf(mn, dpp_from<0x142, 0xA>(pinf, mn));  // row_bcast:15 into rows 1, 3
  mx = __builtin_fmaxf(mx, dpp_from<0x142, 0xA>(ninf, mx));
  mn = __builtin_fminf(mn, dpp_from<0x143, 0xC>(pinf, mn));  // row_bcast:31 into rows 2, 3
  mx = __builtin_fmaxf(mx, dpp_from<0x143, 0xC>(ninf, mx));
  mn = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mn), 63));
  mx = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mx), 63));
}

struct TileArgs {
  GatherArgs g;
  int64_t num_tiles;  // units * 2 * H
};

// Uniform description of one (unit, K|V, head) tile.
struct TileHdr {
  const uint16_t* src;  // cache + layer + head
  uint32_t range;       // bytes from src to the end of the layer's cache slice
  uint8_t* tile;
  uint32_t tile_bytes;  // B * H * D * bits / 8
  uint32_t* scale_word;
  int64_t row0;
  int32_t n_valid, bits, head;
  int32_t page0, page1, page2;  // kUnitPages source pages
};

__device__ __forceinline__ TileHdr tile_header(const GatherArgs& a, const Unit* __restrict__ units, int64_t T) {
  const int64_t per_unit = 2 * int64_t(a.H);
  const int64_t ui = T / per_unit;
  const int32_t rest = int32_t(T - ui * per_unit);
  const int32_t which = rest >= a.H ? 1 : 0;
  const int32_t head = rest - which * a.H;
  const Unit u = units[ui];
  const int tag = u.tag & 0xFF;
  TileHdr h;
  h.src = (which ? a.v_cache : a.k_cache) + int64_t(u.layer) * a.layer_elems + int64_t(head) * a.D;
  h.range = uint32_t((a.layer_elems - int64_t(head) * a.D) * 2);
  h.tile = a.payload + (which ? u.v_off : u.k_off);
  h.scale_word = reinterpret_cast<uint32_t*>(a.scales + u.scale_off + 4 * head + 2 * which);
  h.row0 = u.row0;
  h.n_valid = u.n_valid;
  h.bits = which ? kValueBits[tag] : kKeyBits[tag];
  h.tile_bytes = uint32_t(a.B) * uint32_t(a.H) * uint32_t(a.D) * uint32_t(h.bits) / 8u;
  h.head = head;
  h.page0 = __builtin_amdgcn_readfirstlane(u.page0);
  h.page1 = __builtin_amdgcn_readfirstlane(u.page1);
  h.page2 = __builtin_amdgcn_readfirstlane(u.page2);
  return h;
}

// Cache policy of the tile kernel's buffer loads and stores: non-temporal
// (the intrinsics' cache-policy operand, nt on gfx950).  Cache rows are read
// once and the checkpoint is written once, for a later launch; measured 7%
// faster than the default policy on the 8B-shaped 32-layer write (nt stores
// alone 5%, nt loads alone 2%).
constexpr int kNonTemporal = 2;

// Every lane loads every one of its NL rows; rows past n_valid (and idle
// lanes) read the block's first row instead, so the loads carry no branch and
// stay in flight together.  Offsets are 32-bit from the tile's base (the
// launch checks that a layer's cache slice is below 4 GiB); the buffer range
// check returns zeros past the slice rather than faulting.
template <int NL>
__device__ __forceinline__ void load_tile(const GatherArgs& a, const TileHdr& h, int r, int c, uint4 (&w)[NL]) {
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(h.src), 0, h.range, 0x00020000);
  const uint32_t row_bytes = uint32_t(a.H) * uint32_t(a.D) * 2u;
  const uint32_t slot_mask = (1u << a.log2P) - 1;
  const uint32_t slot0 = uint32_t(h.row0) & slot_mask;  // the block's first row within its first page
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int t = i * a.rpl + r;
    const uint32_t pos = slot0 + uint32_t(t < h.n_valid ? t : 0);  // rows from the first page's start
    const uint32_t k = pos >> a.log2P;                               // 0, 1 or 2
    const uint32_t page = uint32_t(h.page0) + (k >= 1 ? uint32_t(h.page1 - h.page0) : 0u) +
                          (k >= 2 ? uint32_t(h.page2 - h.page1) : 0u);
    const uint32_t off = ((page << a.page_shift) | (pos & slot_mask)) * row_bytes + 16u * uint32_t(c);
    w[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, kNonTemporal));
  }
}

using u32x2 = __attribute__((ext_vector_type(2))) unsigned;
using u32x4 = __attribute__((ext_vector_type(4))) unsigned;
constexpr uint32_t kDropOffset = 0x80000000u;  // past every tile's range: the store is discarded

// The packed word again, opaque to the optimiser, so the range pass's float
// conversions are not kept alive (twice the registers) for the encode pass.
__device__ __forceinline__ uint4 fresh(uint4 w) {
  asm volatile("" : "+v"(w.x), "+v"(w.y), "+v"(w.z), "+v"(w.w));
  return w;
}

// A tile's work in two steps.  tile_range consumes every loaded register
// (the range pass; FP16 tiles are converted in place), so once it returns no
// load of this tile is outstanding and the next tile's loads can be issued
// without the hardware wait counts having to cover them.  tile_store then
// encodes and writes; every store is issued (a lane with nothing to write
// gets an offset past the tile's buffer range, which the hardware drops).
template <bool BF16, int NL>
__device__ __forceinline__ Quant tile_range(const GatherArgs& a, const TileHdr& h, int r, uint4 (&w)[NL],
                                            uint16_t& sb, uint16_t& zb) {
  Quant q;
  if (h.bits == 16) {
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int t = i * a.rpl + r;
      w[i] = t < h.n_valid ? to_half8<BF16>(w[i]) : make_uint4(0, 0, 0, 0);
    }
    sb = zb = 0;
    return q;
  }
  // Every loaded value belongs to the tile (rows past n_valid and idle lanes
  // load rows of the block), so the range runs over all of them unmasked.
  // For bf16 the high value of a word is compared as the raw 32-bit word:
  // its low half only adds less than one bf16 step of magnitude, which never
  // changes the order against another value, and is cleared at the end.
  float mn = __builtin_inff(), mx = -__builtin_inff();
#pragma unroll
  for (int i = 0; i < NL; ++i) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const uint32_t word = word_of(w[i], 2 * p);
      const float x0 = cache_value<BF16>(word, 0);
      const float x1 = BF16 ? __uint_as_float(word) : cache_value<BF16>(word, 1);
      mn = __builtin_fminf(__builtin_fminf(mn, x0), x1);
      mx = __builtin_fmaxf(__builtin_fmaxf(mx, x0), x1);
    }
  }
  wave_range(mn, mx);
  if (BF16) {
    mn = __uint_as_float(__float_as_uint(mn) & 0xFFFF0000u);
    mx = __uint_as_float(__float_as_uint(mx) & 0xFFFF0000u);
  }
  const double qmax = double((1 << h.bits) - 1);
  zb = f16_floor(static_cast<double>(mn) + 0.0);  // -0 counts as +0
  q.zero = f16_value(zb);
  sb = f16_ceil(((static_cast<double>(mx) - q.zero) + 0.0) / qmax);  // -0 span counts as +0
  q.scale = f16_value(sb);
  q.zf = static_cast<float>(q.zero);
  q.invf = q.scale != 0.0 ? static_cast<float>(1.0 / q.scale) : 0.0f;
  q.qmax = uint32_t((1 << h.bits) - 1);
  return q;
}

// STAGE: the workgroup's waves encode every head of one (block, K|V), whose
// code tile [B][H][D] is one contiguous run of the checkpoint.  Each wave
// puts its head's codes into the tile's image in LDS; after a barrier the
// workgroup writes the image out in whole 16-byte lanes, so every 128-byte
// line of the tile is written once, by one store instruction (without it, a
// 4-bit row of one head is half a line, written by a different wave than the
// other half).  FP16 tiles are stored directly either way (each head row is
// whole lines).
template <bool BF16, int NL, bool STAGE>
__device__ __forceinline__ void tile_store(const GatherArgs& a, const TileHdr& h, int r, int c, bool on,
                                           const uint4 (&w)[NL], const Quant& q, uint16_t sb, uint16_t zb,
                                           uint8_t* __restrict__ lds) {
  const uint32_t H = uint32_t(a.H), D = uint32_t(a.D);
  const bool lane0 = (threadIdx.x & 63) == 0;
  const __amdgpu_buffer_rsrc_t out = __builtin_amdgcn_make_buffer_rsrc(h.tile, 0, h.tile_bytes, 0x00020000);
  if (h.bits == 16) {
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int t = i * a.rpl + r;
      const uint32_t off = on && t < a.B ? (uint32_t(t) * H + uint32_t(h.head)) * D * 2 + 16u * uint32_t(c) : kDropOffset;
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, w[i]), out, off, 0, kNonTemporal);
    }
    if (lane0) *h.scale_word = 0u;
    return;
  }
  const bool flat = q.scale == 0.0;  // every value equals the zero: code 0
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int t = i * a.rpl + r;
    const bool valid = t < h.n_valid && !flat;
    const bool store = on && t < a.B;
    const uint4 x = fresh(w[i]);
    if (h.bits == 8) {
      uint2 v = make_uint2(encode_word<BF16, 4>(make_uint4(x.x, x.y, 0, 0), q),
                           encode_word<BF16, 4>(make_uint4(x.z, x.w, 0, 0), q));
      v = valid ? v : make_uint2(0, 0);
      const uint32_t at = (uint32_t(t) * H + uint32_t(h.head)) * D + 8u * uint32_t(c);
      if constexpr (STAGE) {
        if (store) *reinterpret_cast<uint2*>(lds + at) = v;
      } else {
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, v), out, store ? at : kDropOffset, 0,
                                              kNonTemporal);
      }
    } else {
      uint32_t v = encode_word<BF16, 8>(x, q);
      v = valid ? v : 0u;
      const uint32_t at = (uint32_t(t) * H + uint32_t(h.head)) * (D / 2) + 4u * uint32_t(c);
      if constexpr (STAGE) {
        if (store) *reinterpret_cast<uint32_t*>(lds + at) = v;
      } else {
        __builtin_amdgcn_raw_buffer_store_b32(v, out, store ? at : kDropOffset, 0, kNonTemporal);
      }
    }
  }
  if (lane0) *h.scale_word = uint32_t(sb) | (uint32_t(zb) << 16);
  if constexpr (STAGE) {
    __syncthreads();  // every head's codes are in the image
    const uint32_t n16 = h.tile_bytes / 16;
    for (uint32_t i = threadIdx.x; i < n16; i += blockDim.x)
      __builtin_amdgcn_raw_buffer_store_b128(*reinterpret_cast<const u32x4*>(lds + 16 * i), out, 16 * i, 0,
                                             kNonTemporal);
  }
}

template <bool BF16, int NL, bool STAGE>
__global__ __launch_bounds__(kGatherMaxWaves * 64) void gather_tile_kernel(TileArgs s, const Unit* __restrict__ units) {
  extern __shared__ __attribute__((aligned(16))) uint8_t tile_image[];
  const GatherArgs& a = s.g;
  const int lane = threadIdx.x & 63;
  const int r = lane / a.lpr;
  const int c = lane - r * a.lpr;
  const bool on = r < a.rpl;
  const int64_t T =
      xcd_grouped(blockIdx.x, gridDim.x) * (blockDim.x >> 6) + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (T >= s.num_tiles) return;
  const TileHdr h = tile_header(a, units, T);
  uint4 w[NL];
  uint16_t sb, zb;
  load_tile<NL>(a, h, r, c, w);
  const Quant q = tile_range<BF16, NL>(a, h, r, w, sb, zb);
  tile_store<BF16, NL, STAGE>(a, h, r, c, on, w, q, sb, zb, tile_image);
}

// Tiles of 9 to 16 loads per lane (64-token blocks at head_dim 128) as two
// halves on two waves: each wave holds 8 loads (rows [32h, 32h + 32) at
// head_dim 128), the pair exchanges its tile's range through LDS behind the
// workgroup's one barrier, then each wave encodes and stores its half.  An
// 8-wave workgroup holds the two halves of four consecutive tiles.  Held
// whole by one wave, such a tile needs 150 registers and a workgroup per CU;
// as halves it takes 76 (three workgroups per CU), measured 6.6% faster on the
// 70B-shaped write (5488-5494 against 5880-5889 us).  Every wave passes the
// barrier exactly once, FP16 tiles and waves past the last tile included.
constexpr int kHalfWaves = 8;

template <bool BF16>
__global__ __launch_bounds__(kHalfWaves * 64) void gather_half_kernel(TileArgs s, const Unit* __restrict__ units) {
  __shared__ float s_rng[kHalfWaves][2];
  const GatherArgs& a = s.g;
  constexpr int NL = 8;
  const int lane = threadIdx.x & 63;
  const int r = lane / a.lpr;
  const int c = lane - r * a.lpr;
  const bool on = r < a.rpl;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t W = xcd_grouped(blockIdx.x, gridDim.x) * kHalfWaves + wave;
  const int64_t T = W >> 1;
  const int half = int(W & 1);
  const bool live = T < s.num_tiles;  // uniform per wave; every wave still passes the barrier
  const TileHdr h = tile_header(a, units, live ? T : 0);
  const int t_base = half * NL * a.rpl;
  uint4 w[NL];
  {
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(h.src), 0, h.range, 0x00020000);
    const uint32_t row_bytes = uint32_t(a.H) * uint32_t(a.D) * 2u;
    const uint32_t slot_mask = (1u << a.log2P) - 1;
    const uint32_t slot0 = uint32_t(h.row0) & slot_mask;
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int t = t_base + i * a.rpl + r;
      const uint32_t pos = slot0 + uint32_t(t < h.n_valid ? t : 0);
      const uint32_t k = pos >> a.log2P;
      const uint32_t page = uint32_t(h.page0) + (k >= 1 ? uint32_t(h.page1 - h.page0) : 0u) +
                            (k >= 2 ? uint32_t(h.page2 - h.page1) : 0u);
      const uint32_t off = ((page << a.page_shift) | (pos & slot_mask)) * row_bytes + 16u * uint32_t(c);
      w[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, kNonTemporal));
    }
  }
  const uint32_t H = uint32_t(a.H), D = uint32_t(a.D);
  const bool lane0 = lane == 0;
  const __amdgpu_buffer_rsrc_t out = __builtin_amdgcn_make_buffer_rsrc(h.tile, 0, live ? h.tile_bytes : 0u, 0x00020000);
  if (h.bits == 16) {
    __syncthreads();  // matches the range exchange of the other tags (uniform per workgroup)
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int t = t_base + i * a.rpl + r;
      const uint4 v = t < h.n_valid ? to_half8<BF16>(w[i]) : make_uint4(0, 0, 0, 0);
      const uint32_t off = on && t < a.B ? (uint32_t(t) * H + uint32_t(h.head)) * D * 2 + 16u * uint32_t(c) : kDropOffset;
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), out, off, 0, kNonTemporal);
    }
    if (lane0 && half == 0 && live) *h.scale_word = 0u;
    return;
  }
  float mn = __builtin_inff(), mx = -__builtin_inff();
#pragma unroll
  for (int i = 0; i < NL; ++i) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const uint32_t word = word_of(w[i], 2 * p);
      const float x0 = cache_value<BF16>(word, 0);
      const float x1 = BF16 ? __uint_as_float(word) : cache_value<BF16>(word, 1);
      mn = __builtin_fminf(__builtin_fminf(mn, x0), x1);
      mx = __builtin_fmaxf(__builtin_fmaxf(mx, x0), x1);
    }
  }
  wave_range(mn, mx);
  if (lane0) {
    s_rng[wave][0] = mn;
    s_rng[wave][1] = mx;
  }
  __syncthreads();
  mn = __builtin_fminf(mn, s_rng[wave ^ 1][0]);
  mx = __builtin_fmaxf(mx, s_rng[wave ^ 1][1]);
  if (BF16) {
    mn = __uint_as_float(__float_as_uint(mn) & 0xFFFF0000u);
    mx = __uint_as_float(__float_as_uint(mx) & 0xFFFF0000u);
  }
  Quant q;
  const double qmax = double((1 << h.bits) - 1);
  const uint16_t zb = f16_floor(static_cast<double>(mn) + 0.0);
  q.zero = f16_value(zb);
  const uint16_t sb = f16_ceil(((static_cast<double>(mx) - q.zero) + 0.0) / qmax);
  q.scale = f16_value(sb);
  q.zf = static_cast<float>(q.zero);
  q.invf = q.scale != 0.0 ? static_cast<float>(1.0 / q.scale) : 0.0f;
  q.qmax = uint32_t((1 << h.bits) - 1);
  const bool flat = q.scale == 0.0;
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int t = t_base + i * a.rpl + r;
    const bool valid = t < h.n_valid && !flat;
    const bool store = on && t < a.B;
    const uint4 x = fresh(w[i]);
    if (h.bits == 8) {
      uint2 v = make_uint2(encode_word<BF16, 4>(make_uint4(x.x, x.y, 0, 0), q),
                           encode_word<BF16, 4>(make_uint4(x.z, x.w, 0, 0), q));
      v = valid ? v : make_uint2(0, 0);
      const uint32_t at = (uint32_t(t) * H + uint32_t(h.head)) * D + 8u * uint32_t(c);
      __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, v), out, store ? at : kDropOffset, 0, kNonTemporal);
    } else {
      uint32_t v = encode_word<BF16, 8>(x, q);
      v = valid ? v : 0u;
      const uint32_t at = (uint32_t(t) * H + uint32_t(h.head)) * (D / 2) + 4u * uint32_t(c);
      __builtin_amdgcn_raw_buffer_store_b32(v, out, store ? at : kDropOffset, 0, kNonTemporal);
    }
  }
  if (lane0 && half == 0 && live) *h.scale_word = uint32_t(sb) | (uint32_t(zb) << 16);
}

// The staged store needs a workgroup to hold exactly the heads of one
// (block, K|V) -- one wave per head -- and the 8-bit image of a tile in LDS.
constexpr uint32_t kTileImageMax = 64u << 10;

template <bool BF16, int NL>
hipError_t launch_tile_nl(const TileArgs& s, const Unit* units, int wg, uint32_t image, hipStream_t stream) {
  const int64_t waves = wg / 64;
  const dim3 grid(static_cast<uint32_t>((s.num_tiles + waves - 1) / waves));
  if (image)
    hipLaunchKernelGGL((gather_tile_kernel<BF16, NL, true>), grid, dim3(wg), image, stream, s, units);
  else
    hipLaunchKernelGGL((gather_tile_kernel<BF16, NL, false>), grid, dim3(wg), 0, stream, s, units);
  return hipGetLastError();
}

template <bool BF16>
hipError_t launch_tile(const TileArgs& s, const Unit* units, int nl, int wg, uint32_t image, hipStream_t stream) {
  switch (nl) {
    case 2: return launch_tile_nl<BF16, 2>(s, units, wg, image, stream);
    case 4: return launch_tile_nl<BF16, 4>(s, units, wg, image, stream);
    case 8: return launch_tile_nl<BF16, 8>(s, units, wg, image, stream);
    default: {
      const dim3 grid(static_cast<uint32_t>((2 * s.num_tiles + kHalfWaves - 1) / kHalfWaves));
      hipLaunchKernelGGL((gather_half_kernel<BF16>), grid, dim3(kHalfWaves * 64), 0, stream, s, units);
      return hipGetLastError();
    }
  }
}

template <bool BF16>
void launch_gather(const GatherArgs& a, int nl, dim3 grid, dim3 block, hipStream_t stream) {
  switch (nl) {
    case 2: hipLaunchKernelGGL((gather_kernel<BF16, 2>), grid, block, 0, stream, a); break;
    case 4: hipLaunchKernelGGL((gather_kernel<BF16, 4>), grid, block, 0, stream, a); break;
    case 8: hipLaunchKernelGGL((gather_kernel<BF16, 8>), grid, block, 0, stream, a); break;
    default: hipLaunchKernelGGL((gather_kernel<BF16, 16>), grid, block, 0, stream, a); break;
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
  if (reinterpret_cast<uintptr_t>(payload) % 16 || reinterpret_cast<uintptr_t>(scales) % 8)
    return PKV_ERR_INVALID_ARGUMENT;
  if (payload_bytes < info.payload_bytes || scale_bytes < info.scale_bytes || cache_bytes < info.cache_bytes)
    return PKV_ERR_INVALID_ARGUMENT;
  const uint64_t pb = info.payload_bytes, sb = info.scale_bytes;
  pkv::ByteRange caches[2];
  int n = 0;
  if (!pkv::cache_ranges(plan->host.model, k_cache, v_cache, info.cache_bytes, caches, n))
    return PKV_ERR_INVALID_ARGUMENT;
  if (pkv::overlap(payload, pb, scales, sb)) return PKV_ERR_INVALID_ARGUMENT;
  for (int i = 0; i < n; ++i)
    if (pkv::overlap(payload, pb, caches[i].p, caches[i].n) || pkv::overlap(scales, sb, caches[i].p, caches[i].n))
      return PKV_ERR_INVALID_ARGUMENT;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != plan->device) return PKV_ERR_DEVICE;
  // The old caches must be device memory of the plan's device; the
  // checkpoint may also go to pinned host memory, written through its device
  // mapping.  Anything else would fault in the kernel.
  const void *p_dev = nullptr, *s_dev = nullptr;
  pkv_status_t st;
  if ((st = pkv::device_resident(plan, k_cache)) != PKV_OK || (st = pkv::device_resident(plan, v_cache)) != PKV_OK ||
      (st = pkv::kernel_accessible(plan, payload, &p_dev)) != PKV_OK ||
      (st = pkv::kernel_accessible(plan, scales, &s_dev)) != PKV_OK)
    return st;

  const pkv_model_t& m = plan->host.model;
  pkv::GatherArgs a;
  a.units = plan->d_units;
  a.page_tables = plan->d_page_tables;
  a.k_cache = static_cast<const uint16_t*>(k_cache);
  a.v_cache = static_cast<const uint16_t*>(v_cache);
  a.payload = static_cast<uint8_t*>(const_cast<void*>(p_dev));
  a.scales = static_cast<uint16_t*>(const_cast<void*>(s_dev));
  a.layer_elems = pkv::layer_elems(m);
  a.page_shift = pkv::page_shift(m);
  a.H = m.num_kv_heads;
  a.D = m.head_dim;
  a.B = m.block_tokens;
  a.log2P = plan->host.log2_page;
  a.lpr = m.head_dim / 8;
  a.rpl = 64 / a.lpr;
  const int nload = (m.block_tokens + a.rpl - 1) / a.rpl;  // loads per lane covering a block
  const int nl = pkv::gather_loads_per_chunk(nload);
  a.nchunk = (nload + nl - 1) / nl;
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  if (a.nchunk == 1 && m.block_tokens <= 2 * m.page_size + 1 && a.layer_elems * 2 < (int64_t(1) << 32)) {
    // Tiles of at most 16 loads per lane on at most kUnitPages pages, layer
    // slices below 4 GiB: the tile kernel (up to 8 loads) or the half-tile
    // kernel (9 to 16).
    pkv::TileArgs sa;
    sa.g = a;
    sa.num_tiles = info.num_units * 2 * m.num_kv_heads;
    // Staged stores when a workgroup is one wave per head of one (block, K|V)
    // of at most 8 loads per lane.  (Larger tiles staged whole in a
    // workgroup per CU ran 18-20% slower on the 70B-shaped write: the barrier
    // left the CU without loads in flight while it wrote.)
    const uint64_t image = uint64_t(m.block_tokens) * m.num_kv_heads * m.head_dim;
    const uint32_t stage =
        nl <= 8 && plan->host.workgroup == 64 * m.num_kv_heads && image <= pkv::kTileImageMax ? uint32_t(image) : 0;
    const hipError_t e = m.out_dtype == PKV_OUT_BF16
                             ? pkv::launch_tile<true>(sa, plan->d_units, nl, plan->host.workgroup, stage, stream)
                             : pkv::launch_tile<false>(sa, plan->d_units, nl, plan->host.workgroup, stage, stream);
    return e == hipSuccess ? PKV_OK : PKV_ERR_DEVICE;
  }
  const dim3 grid(static_cast<uint32_t>(2 * info.num_units)), block(plan->host.workgroup);
  if (m.out_dtype == PKV_OUT_BF16)
    pkv::launch_gather<true>(a, nl, grid, block, stream);
  else
    pkv::launch_gather<false>(a, nl, grid, block, stream);
  return hipGetLastError() == hipSuccess ? PKV_OK : PKV_ERR_DEVICE;
}

}  // extern "C"
