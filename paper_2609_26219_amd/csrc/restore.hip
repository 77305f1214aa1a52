// Device half of libpkv: the fused dequantize / RoPE-correct / scatter kernel
// of the suffix restore (PatchKV Section IV-D, Eq. 3, Eq. 14) for gfx950,
// and the C entry points that own device memory and launch it.
//
// Work decomposition.  One workgroup restores one unit: every head of up to
// 16K output elements' worth of consecutive tokens of one reused block of
// one layer that share one cache page (at 8 heads x 128 and 16-token pages,
// the block's rows in each page it touches).  The unit's K rows and V rows
// are contiguous in the payload (token-major tiles) and each token lands on
// one cache slot whose H*D elements are contiguous, so a unit is a streaming
// row-to-row transform.  A thread owns a fixed piece of every row it
// touches: channels [8j, 8j+8) and [D/2+8j, D/2+8j+8) of one head.  For keys
// that is a set of whole rotary pairs, so the rotation needs no cross-lane
// exchange; for keys and values alike, each store instruction of a wave
// writes whole 128-byte lines.  Threads (t0, c), c = head*(D/16) + j, own
// tokens t0, t0+tpp, ... with tpp = threads / (H*D/16) (at most four of
// them; a workgroup has 64 to 256 threads, restore_workgroup())
// and issue the loads of all their tokens before the first store; the
// unit's one page comes with its work item, so no workgroup-wide staging or
// barrier is needed except for the per-request cos/sin table (staged before
// the payload loads or after them: the two start orders of Stage).  An LDS claim caps
// the workgroups sharing a compute unit at two to four, chosen per plan from
// its read:write byte ratio, its unit size, whether its keys rotate and the
// cache layout (restore_workgroups_per_cu).
//
// Cache layouts.  With separate caches a page's K slots and V slots sit in
// two buffers; with paired pages they are one contiguous run, K then V.
// Both are addressed as page << page_shift slot rows from the layer's start.
//
// Arithmetic.  Codes decode exactly.  Keys are rotated in double precision
// (v_fma_f64 issues at the rate of a non-packed v_fma_f32 on CDNA4, and
// packed f32 is off in this build; an f32 rotation measured no faster) with
// a double (cos, sin) table, so the rotated value
// carries ~2^-53 relative error even under cancellation; values use one
// single-precision FMA.  Results go to float, then to the cache dtype with
// the hardware round-to-nearest-even conversions.
//
// Memory behaviour (8B-shaped 32K-token workload, measured): the kernel
// moves 1.0025x the algorithmic bytes; the write-heavy mixed stream bounds it,
// and paired pages let the memory system stream the writes faster.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <new>

#include "pkv.h"
#include "pkv_internal.h"

namespace pkv {
namespace {

// Register budget for four waves per SIMD, so that the (cos, sin) pairs and
// four tokens' payload of a thread stay in registers (the residency cap then
// keeps two to four).
constexpr int kMinWavesPerEU = 4;

// Launches of at most this many rounds of resident workgroups take the late
// start order of the restore kernel (see Stage).
constexpr int64_t kLateRounds = 6;

struct KernelArgs {
  const Unit* units;
  const double* tables;
  const uint8_t* payload;
  const uint16_t* scales;
  uint16_t* k_cache;
  uint16_t* v_cache;
  int64_t layer_elems;  // elements of one layer of a cache: pool_pages * P * H * D, twice that when paired
  int32_t H, D, log2P, cols, tpp;
  int32_t cols_shift, dq_shift;  // log2 of cols and of D/16 when they are powers of two, else -1
  int32_t R;            // rotary channels per head
  int32_t page_shift;   // slot rows from a layer's start to page p: p << page_shift
  // Units whose K rows start outside [win_lo, win_hi) payload bytes are
  // skipped (the staged restore runs a request's layer in payload windows);
  // [0, 2^64) everywhere else.
  uint64_t win_lo, win_hi;
};

__device__ __forceinline__ float half_bits_to_float(uint32_t h) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(h)));
}

// double -> float with the hardware conversion.  The empty asm pins the
// float: without it the compiler merges double -> float -> half/bf16 into one
// software double -> half/bf16 rounding of 10-40 integer instructions.
__device__ __forceinline__ float to_float(double d) {
  float f = static_cast<float>(d);
  asm volatile("" : "+v"(f));
  return f;
}

// Loads and stores are buffer instructions: a unit's payload runs and its
// destination page are uniform bases (scalar registers), each thread keeps
// one 32-bit offset per run, and a thread's later tokens add a uniform
// scalar offset -- no per-access 64-bit address arithmetic.  A page of one
// cache is at most 2 GiB (checked at plan time), so offsets fit 32 bits.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
// A buffer of `bytes` bytes from `base`: loads past its end return 0 and
// stores past it are dropped by the hardware, with no memory access.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
}
constexpr uint32_t kWholeRange = 0xFFFFFFFFu;
// An offset past every bounded buffer of the kernel (a cache page is below
// 2 GiB, a unit's payload run a few MiB): accesses there are dropped.
constexpr uint32_t kOutside = 0x80000000u;
// Cache-policy operand of the buffer intrinsics: nt (non-temporal) on gfx950.
constexpr int kNonTemporal = 2;

// Restored rows are written once and not read again by this launch: store
// them non-temporally (measured 2% faster on the 8B-shaped workload).
//
// The whole offset goes in the VGPR operand and the SGPR offset is 0.  A
// 16-byte store reads its data registers after it issues, so an instruction
// right behind it must not overwrite them; the compiler inserts the wait
// state for that only when the store's SGPR offset is a constant, and with
// a register SGPR offset gfx950 was seen storing the next instruction's
// result (a token's 16 outputs replaced, now and then, by an address or a
// decoded value).
__device__ __forceinline__ void store_row_piece(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, uint4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, voff + soff, 0, kNonTemporal);
}

// Two floats to two bfloat16 / binary16 values, round to nearest even, in
// one packed conversion (v_cvt_pk_bf16_f32 / v_cvt_pk_f16_f32 on gfx950;
// converting each value alone takes a conversion each plus a shift and an or).
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
template <bool BF16>
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  const f32x2 v = {a, b};
  if constexpr (BF16) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
  } else {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, f16x2));
  }
}

template <bool BF16>
__device__ __forceinline__ uint4 pack8(const float* v) {
  return make_uint4(pack2<BF16>(v[0], v[1]), pack2<BF16>(v[2], v[3]), pack2<BF16>(v[4], v[5]),
                    pack2<BF16>(v[6], v[7]));
}

// Eight channel codes / values of one half-row piece, as integers (codes) or
// binary16 bit patterns (FP16 tag).
template <int BITS>
struct Chunk8;
template <>
struct Chunk8<16> {
  uint4 w;
  // FP16 runs load non-temporally: 1.4% faster on an all-FP16 checkpoint
  // (code runs measured 2-3% slower that way, so they keep the default).
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    w = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kNonTemporal));
  }
  __device__ __forceinline__ uint32_t raw(int e) const {
    const uint32_t word = e < 2 ? w.x : e < 4 ? w.y : e < 6 ? w.z : w.w;
    return (word >> (16 * (e & 1))) & 0xFFFFu;
  }
};
template <>
struct Chunk8<8> {
  uint2 w;
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    w = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
  }
  __device__ __forceinline__ uint32_t raw(int e) const { return ((e < 4 ? w.x : w.y) >> (8 * (e & 3))) & 0xFFu; }
};
template <>
struct Chunk8<4> {
  uint32_t w;
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    w = __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0);
  }
  // Element 2k is the low nibble of byte k, element 2k + 1 its high nibble:
  // mask the word into four byte-wide codes of each parity, so each code
  // converts with one v_cvt_f32_ubyte (no bit-field extract per code).
  __device__ __forceinline__ uint32_t raw(int e) const {
    const uint32_t bytes = (e & 1 ? w >> 4 : w) & 0x0F0F0F0Fu;
    return (bytes >> (8 * (e >> 1))) & 0xFFu;
  }
};

// Decode element e of a chunk to float (exact for codes <= 255 and binary16).
template <int BITS>
__device__ __forceinline__ float decode_f(const Chunk8<BITS>& c, int e, float s, float z) {
  if constexpr (BITS == 16) {
    return half_bits_to_float(c.raw(e));
  } else {
    return __builtin_fmaf(static_cast<float>(c.raw(e)), s, z);
  }
}

template <int BITS>
__device__ __forceinline__ double decode_d(const Chunk8<BITS>& c, int e, double s, double z) {
  if constexpr (BITS == 16) {
    return static_cast<double>(half_bits_to_float(c.raw(e)));
  } else {
    return __builtin_fma(static_cast<double>(c.raw(e)), s, z);
  }
}

// Key piece j of a head: two runs of 8 channels, at `lo` and `hi`, and
// whether each run rotates.  Rotate-half (pairs (i, i + R/2)): piece j < R/16
// holds channels [8j, 8j+8) and [R/2 + 8j, ...), element e pairing with
// element e; pieces past R/16 hold pass-through channels [R, D) in the same
// two-halves arrangement.  Interleaved (pairs (2i, 2i+1)): piece j holds
// [8j, 8j+8) and [D/2 + 8j, ...), each pairing elements 2k and 2k+1; a run
// rotates when it lies inside [0, R).  The (cos, sin) table is laid out by
// the planner in the same element order.
struct KeyPiece {
  int lo, hi;
  bool rot_lo, rot_hi;
};

template <int STYLE>
__device__ __forceinline__ KeyPiece key_piece(int j, int D, int R) {
  KeyPiece p;
  if constexpr (STYLE == PKV_ROPE_HALF) {
    if (8 * j < R / 2) {
      p.lo = 8 * j;
      p.hi = R / 2 + 8 * j;
      p.rot_lo = p.rot_hi = true;
    } else {
      const int q = j - R / 16;
      p.lo = R + 8 * q;
      p.hi = R + (D - R) / 2 + 8 * q;
      p.rot_lo = p.rot_hi = false;
    }
  } else {
    p.lo = 8 * j;
    p.hi = D / 2 + 8 * j;
    p.rot_lo = p.lo + 8 <= R;
    p.rot_hi = p.hi + 8 <= R;
  }
  return p;
}

// Rotate one interleaved run: pairs (2k, 2k+1) with cs[k].
template <int KBITS>
__device__ __forceinline__ void rotate_pairs(const Chunk8<KBITS>& c, double s64, double z64,
                                             const double2* __restrict__ cs, float* out) {
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const double x = decode_d<KBITS>(c, 2 * k, s64, z64);
    const double y = decode_d<KBITS>(c, 2 * k + 1, s64, z64);
    out[2 * k] = to_float(__builtin_fma(x, cs[k].x, -(y * cs[k].y)));
    out[2 * k + 1] = to_float(__builtin_fma(y, cs[k].x, x * cs[k].y));
  }
}

template <int KBITS>
__device__ __forceinline__ void decode_run(const Chunk8<KBITS>& c, float s, float z, float* out) {
#pragma unroll
  for (int e = 0; e < 8; ++e) out[e] = decode_f<KBITS>(c, e, s, z);
}

// Keys of one (token, head), piece p, from its two loaded runs: decode,
// rotate, round, store.
template <int KBITS, bool ROT, int STYLE, bool BF16>
__device__ __forceinline__ void key_store(const Chunk8<KBITS>& lo, const Chunk8<KBITS>& hi, const KeyPiece& p, float ks,
                                          float kz, const double2* __restrict__ cs, __amdgpu_buffer_rsrc_t dst,
                                          uint32_t doff, uint32_t soff) {
  uint4 out_lo, out_hi;
  if constexpr (KBITS == 16 && !ROT && !BF16) {
    // binary16 in, binary16 out, no rotation: the bits are the result.
    out_lo = lo.w;
    out_hi = hi.w;
  } else {
    float a[8], b[8];
    if constexpr (ROT && STYLE == PKV_ROPE_HALF) {
      if (p.rot_lo) {
        const double s64 = ks, z64 = kz;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const double x = decode_d<KBITS>(lo, e, s64, z64);
          const double y = decode_d<KBITS>(hi, e, s64, z64);
          a[e] = to_float(__builtin_fma(x, cs[e].x, -(y * cs[e].y)));
          b[e] = to_float(__builtin_fma(y, cs[e].x, x * cs[e].y));
        }
      } else {
        decode_run<KBITS>(lo, ks, kz, a);
        decode_run<KBITS>(hi, ks, kz, b);
      }
    } else if constexpr (ROT) {  // interleaved
      if (p.rot_lo)
        rotate_pairs<KBITS>(lo, ks, kz, cs, a);
      else
        decode_run<KBITS>(lo, ks, kz, a);
      if (p.rot_hi)
        rotate_pairs<KBITS>(hi, ks, kz, cs + 4, b);
      else
        decode_run<KBITS>(hi, ks, kz, b);
    } else {
      decode_run<KBITS>(lo, ks, kz, a);
      decode_run<KBITS>(hi, ks, kz, b);
    }
    out_lo = pack8<BF16>(a);
    out_hi = pack8<BF16>(b);
  }
  store_row_piece(dst, doff + 2 * p.lo, soff, out_lo);
  store_row_piece(dst, doff + 2 * p.hi, soff, out_hi);
}

// Values of one (token, head), piece j (never rotated).
template <int VBITS, bool BF16>
__device__ __forceinline__ void value_store(const Chunk8<VBITS>& lo, const Chunk8<VBITS>& hi, int j, int D, float vs,
                                            float vz, __amdgpu_buffer_rsrc_t dst, uint32_t doff, uint32_t soff) {
  uint4 out_lo, out_hi;
  if constexpr (VBITS == 16 && !BF16) {
    out_lo = lo.w;
    out_hi = hi.w;
  } else {
    float a[8], b[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      a[e] = decode_f<VBITS>(lo, e, vs, vz);
      b[e] = decode_f<VBITS>(hi, e, vs, vz);
    }
    out_lo = pack8<BF16>(a);
    out_hi = pack8<BF16>(b);
  }
  store_row_piece(dst, doff + 16 * j, soff, out_lo);
  store_row_piece(dst, doff + D + 16 * j, soff, out_hi);
}

// What a thread needs for every token of its unit.
struct Piece {
  int head, j;
  KeyPiece kp;
  float ks, kz, vs, vz;
  __amdgpu_buffer_rsrc_t kdst, vdst;  // the unit's destination page in each cache
  uint32_t doff;                      // bytes from the page's start to the thread's first token, its head
};

// Two orders of a workgroup's start, chosen per launch (launch_restore).
//
// Early (deep launches of 256-thread workgroups): the request's (cos, sin)
// table is staged in LDS behind a barrier at the start, then each thread
// loads its head's scales, then issues its payload loads.  Other resident
// workgroups hide that chain of dependent loads.
//
// Late (launches a few rounds of resident workgroups deep, and narrow rows,
// where too little other work hides it): table entry tid and the head's
// scale word are loaded at the
// start, the payload loads are issued right after, and only then are the
// table entries written to LDS, the barrier passed and the scales
// converted.  The table, the scales and the payload are then in flight
// together: one memory latency before the first store instead of three.
// Every wave passes the barrier exactly once, as the token-count switch is
// wave-uniform in this order (restore_unit).
struct Stage {
  double* s_tab;        // LDS, D doubles
  const double* table;  // the request's table in global memory
  double tval;          // entry tid (threads < D)
  uint2 sw;             // the thread's head: K scale, K zero, V scale, V zero (binary16)
  bool pending;         // not yet staged (uniform across the workgroup)
  int tid, D, threads;
};

template <int TAG, bool ROT>
__device__ __forceinline__ void finish_stage(Stage& st, Piece& q, double2* cs) {
  if (!st.pending) return;
  if constexpr (ROT) {
    if (st.tid < st.D) st.s_tab[st.tid] = st.tval;
    for (int i = st.tid + st.threads; i < st.D; i += st.threads) st.s_tab[i] = st.table[i];
    __syncthreads();
#pragma unroll
    for (int e = 0; e < 8; ++e) cs[e] = *reinterpret_cast<const double2*>(st.s_tab + 2 * (8 * q.j + e));
  }
  if constexpr (TAG != PKV_TAG_FP16) {
    uint2 sw = st.sw;
    asm volatile("" : "+v"(sw.x), "+v"(sw.y));  // keeps the conversion behind the payload loads
    q.ks = half_bits_to_float(sw.x & 0xFFFFu);
    q.kz = half_bits_to_float(sw.x >> 16);
    q.vs = half_bits_to_float(sw.y & 0xFFFFu);
    q.vz = half_bits_to_float(sw.y >> 16);
  }
  st.pending = false;
}

// NK tokens of one thread (t, t + tpp, ...): every load is issued before the
// first store, so a wave keeps NK tokens of payload in flight.  No load
// depends on another: the unit's page comes with its work item.  Token k of
// the thread is k * tpp rows further in the payload and in the page.  In the
// late order only the first `valid` tokens are real: the accesses of the
// others get offsets past their buffers, which the hardware drops.
template <int NK, int TAG, bool ROT, int STYLE, bool BF16, bool LATE>
__device__ __forceinline__ void restore_tokens(const KernelArgs& a, const Unit& u, int t, Piece& q,
                                               double2* __restrict__ cs, Stage& st, int valid) {
  constexpr int KB = kKeyBits[TAG];
  constexpr int VB = kValueBits[TAG];
  const uint32_t H = uint32_t(a.H), D = uint32_t(a.D), tpp = uint32_t(a.tpp);
  const uint32_t rows = uint32_t(u.n_valid) * H;
  const __amdgpu_buffer_rsrc_t kr = raw_rsrc(a.payload + u.k_off, LATE ? rows * (D * KB / 8) : kWholeRange);
  const __amdgpu_buffer_rsrc_t vr = raw_rsrc(a.payload + u.v_off, LATE ? rows * (D * VB / 8) : kWholeRange);
  const uint32_t row = uint32_t(t) * H + uint32_t(q.head);  // the thread's first (token, head) row of the unit
  const uint32_t k_lo = row * (D * KB / 8) + uint32_t(q.kp.lo) * KB / 8;
  const uint32_t k_hi = row * (D * KB / 8) + uint32_t(q.kp.hi) * KB / 8;
  const uint32_t v_lo = row * (D * VB / 8) + uint32_t(8 * q.j) * VB / 8;
  const uint32_t v_hi = v_lo + (D / 2) * VB / 8;
  const uint32_t doff = q.doff + uint32_t(t) * H * D * 2;
  Chunk8<KB> klo[NK], khi[NK];
  Chunk8<VB> vlo[NK], vhi[NK];
#pragma unroll
  for (int k = 0; k < NK; ++k) {
    const bool on = !LATE || k < valid;
    klo[k].load(kr, on ? k_lo : kOutside, k * tpp * H * D * KB / 8);
    khi[k].load(kr, on ? k_hi : kOutside, k * tpp * H * D * KB / 8);
    vlo[k].load(vr, on ? v_lo : kOutside, k * tpp * H * D * VB / 8);
    vhi[k].load(vr, on ? v_hi : kOutside, k * tpp * H * D * VB / 8);
  }
  if constexpr (LATE) finish_stage<TAG, ROT>(st, q, cs);
#pragma unroll
  for (int k = 0; k < NK; ++k) {
    const uint32_t d = !LATE || k < valid ? doff : kOutside;
    key_store<KB, ROT, STYLE, BF16>(klo[k], khi[k], q.kp, q.ks, q.kz, cs, q.kdst, d, k * tpp * H * D * 2);
    value_store<VB, BF16>(vlo[k], vhi[k], q.j, D, q.vs, q.vz, q.vdst, d, k * tpp * H * D * 2);
  }
}

template <int TAG, bool ROT, int STYLE, bool BF16, bool LATE>
__device__ __forceinline__ void restore_unit(const KernelArgs& a, const Unit& u, const double* __restrict__ s_tab,
                                             Stage& st, int t0, int head, int j) {
  Piece q;
  q.head = head;
  q.j = j;
  q.kp = key_piece<STYLE>(j, a.D, a.R);
  q.ks = q.kz = q.vs = q.vz = 0.f;
  if constexpr (TAG != PKV_TAG_FP16 && !LATE) {
    const uint2 sw = *reinterpret_cast<const uint2*>(a.scales + u.scale_off + 4 * head);
    q.ks = half_bits_to_float(sw.x & 0xFFFFu);
    q.kz = half_bits_to_float(sw.x >> 16);
    q.vs = half_bits_to_float(sw.y & 0xFFFFu);
    q.vz = half_bits_to_float(sw.y >> 16);
  }
  // A unit's rows share one page, carried in its work item.
  const int64_t page = int64_t(u.layer) * a.layer_elems + (int64_t(u.page1) << a.page_shift) * (int64_t(a.H) * a.D);
  q.kdst = raw_rsrc(a.k_cache + page, LATE ? kOutside : kWholeRange);
  q.vdst = raw_rsrc(a.v_cache + page, LATE ? kOutside : kWholeRange);
  q.doff = (uint32_t(u.row0 & ((int64_t(1) << a.log2P) - 1)) * uint32_t(a.H) + uint32_t(head)) * uint32_t(a.D) * 2;
  double2 cs[8];  // (cos, sin) of this thread's eight rotary pairs
  if constexpr (ROT && !LATE) {
#pragma unroll
    for (int e = 0; e < 8; ++e) cs[e] = *reinterpret_cast<const double2*>(s_tab + 2 * (8 * j + e));
  }
  // A unit holds at most 4 * tpp tokens when H*D divides 4096, so a thread
  // has at most four; FP16 runs them two at a time (16-byte runs take twice
  // the registers).  Other shapes take the remaining tokens one by one.
  if constexpr (!LATE) {
    const int nk = t0 < u.n_valid ? (u.n_valid - t0 + a.tpp - 1) / a.tpp : 0;
    if constexpr (TAG != PKV_TAG_FP16) {
      switch (nk) {
        case 0: return;
        case 1: restore_tokens<1, TAG, ROT, STYLE, BF16, false>(a, u, t0, q, cs, st, 1); return;
        case 2: restore_tokens<2, TAG, ROT, STYLE, BF16, false>(a, u, t0, q, cs, st, 2); return;
        case 3: restore_tokens<3, TAG, ROT, STYLE, BF16, false>(a, u, t0, q, cs, st, 3); return;
        case 4: restore_tokens<4, TAG, ROT, STYLE, BF16, false>(a, u, t0, q, cs, st, 4); return;
        default: break;
      }
    } else if (nk <= 4) {
      for (int k = nk, t = t0; k > 0; k -= 2, t += 2 * a.tpp) {
        if (k >= 2)
          restore_tokens<2, TAG, ROT, STYLE, BF16, false>(a, u, t, q, cs, st, 2);
        else
          restore_tokens<1, TAG, ROT, STYLE, BF16, false>(a, u, t, q, cs, st, 1);
      }
      return;
    }
    for (int t = t0; t < u.n_valid; t += a.tpp) restore_tokens<1, TAG, ROT, STYLE, BF16, false>(a, u, t, q, cs, st, 1);
  } else {
    // Late order: the switch takes lane 0's count, the largest in its wave
    // (lanes are in token order; threads past tpp rows count 0), so each
    // wave takes one case and passes the staging barrier once.
    const int nk_t = t0 < a.tpp && t0 < u.n_valid ? (u.n_valid - t0 + a.tpp - 1) / a.tpp : 0;
    const int nk = __builtin_amdgcn_readfirstlane(nk_t);
    if constexpr (TAG != PKV_TAG_FP16) {
      switch (nk) {
        case 0: finish_stage<TAG, ROT>(st, q, cs); return;
        case 1: restore_tokens<1, TAG, ROT, STYLE, BF16, true>(a, u, t0, q, cs, st, nk_t); return;
        case 2: restore_tokens<2, TAG, ROT, STYLE, BF16, true>(a, u, t0, q, cs, st, nk_t); return;
        case 3: restore_tokens<3, TAG, ROT, STYLE, BF16, true>(a, u, t0, q, cs, st, nk_t); return;
        case 4: restore_tokens<4, TAG, ROT, STYLE, BF16, true>(a, u, t0, q, cs, st, nk_t); return;
        default: break;
      }
    } else {
      const int t2 = t0 + 2 * a.tpp;
      switch (nk) {
        case 0: finish_stage<TAG, ROT>(st, q, cs); return;
        case 1: restore_tokens<1, TAG, ROT, STYLE, BF16, true>(a, u, t0, q, cs, st, nk_t); return;
        case 2: restore_tokens<2, TAG, ROT, STYLE, BF16, true>(a, u, t0, q, cs, st, nk_t); return;
        case 3:
          restore_tokens<2, TAG, ROT, STYLE, BF16, true>(a, u, t0, q, cs, st, nk_t);
          restore_tokens<1, TAG, ROT, STYLE, BF16, true>(a, u, t2, q, cs, st, nk_t - 2);
          return;
        case 4:
          restore_tokens<2, TAG, ROT, STYLE, BF16, true>(a, u, t0, q, cs, st, nk_t);
          restore_tokens<2, TAG, ROT, STYLE, BF16, true>(a, u, t2, q, cs, st, nk_t - 2);
          return;
        default: break;
      }
    }
    finish_stage<TAG, ROT>(st, q, cs);
    if (t0 < a.tpp)
      for (int t = t0; t < u.n_valid; t += a.tpp) restore_tokens<1, TAG, ROT, STYLE, BF16, true>(a, u, t, q, cs, st, 1);
  }
}

template <bool BF16, int STYLE, bool LATE>
__global__ __launch_bounds__(kWorkgroup, kMinWavesPerEU) void restore_kernel(KernelArgs a) {
  __shared__ __attribute__((aligned(16))) double s_tab[kMaxHeadDim];
  const Unit u = a.units[xcd_grouped(blockIdx.x, gridDim.x)];
  if (u.k_off < a.win_lo || u.k_off >= a.win_hi) return;  // uniform across the workgroup
  const int tid = threadIdx.x;
  const int tag = u.tag & 0xFF;
  const bool rot = (u.tag & kUnitRotate) != 0;
  // Thread -> (token, head, piece): shifts when the row's piece counts are
  // powers of two (uniform branches), divisions otherwise.
  const int t0 = a.cols_shift >= 0 ? tid >> a.cols_shift : tid / a.cols;
  const int c = tid - t0 * a.cols;
  const int dq = a.D >> 4;
  const int head = a.dq_shift >= 0 ? c >> a.dq_shift : c / dq;
  const int j = c - head * dq;
  Stage st;
  if constexpr (LATE) {
    // Threads past tpp token rows have no tokens but take part in the barrier.
    st.s_tab = s_tab;
    st.table = a.tables + u.table_off;
    st.tid = tid;
    st.D = a.D;
    st.threads = int(blockDim.x);
    st.pending = true;
    st.tval = rot && tid < a.D ? st.table[tid] : 0.0;
    st.sw = tag != PKV_TAG_FP16 ? *reinterpret_cast<const uint2*>(a.scales + u.scale_off + 4 * head) : make_uint2(0, 0);
  } else {
    if (rot) {  // uniform across the workgroup
      for (int i = tid; i < a.D; i += int(blockDim.x)) s_tab[i] = a.tables[u.table_off + i];
      __syncthreads();
    }
    if (t0 >= a.tpp) return;
  }
  switch (tag * 2 + (rot ? 1 : 0)) {
    case 0: restore_unit<PKV_TAG_FP16, false, STYLE, BF16, LATE>(a, u, s_tab, st, t0, head, j); break;
    case 1: restore_unit<PKV_TAG_FP16, true, STYLE, BF16, LATE>(a, u, s_tab, st, t0, head, j); break;
    case 2: restore_unit<PKV_TAG_K8V8, false, STYLE, BF16, LATE>(a, u, s_tab, st, t0, head, j); break;
    case 3: restore_unit<PKV_TAG_K8V8, true, STYLE, BF16, LATE>(a, u, s_tab, st, t0, head, j); break;
    case 4: restore_unit<PKV_TAG_K8V4, false, STYLE, BF16, LATE>(a, u, s_tab, st, t0, head, j); break;
    case 5: restore_unit<PKV_TAG_K8V4, true, STYLE, BF16, LATE>(a, u, s_tab, st, t0, head, j); break;
    case 6: restore_unit<PKV_TAG_K4V4, false, STYLE, BF16, LATE>(a, u, s_tab, st, t0, head, j); break;
    default: restore_unit<PKV_TAG_K4V4, true, STYLE, BF16, LATE>(a, u, s_tab, st, t0, head, j); break;
  }
}

bool ranges_overlap(const void* a, uint64_t na, const void* b, uint64_t nb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}

}  // namespace
}  // namespace pkv

namespace pkv {

pkv_status_t upload_plan(HostPlan&& hp, pkv_plan** out) {
  *out = nullptr;
  pkv_plan* plan = new (std::nothrow) pkv_plan();
  if (!plan) return PKV_ERR_OUT_OF_MEMORY;
  plan->host = std::move(hp);
  // One allocation, 256-byte aligned sections.
  auto al = [](size_t x) { return (x + 255) & ~size_t(255); };
  const size_t n_units = plan->host.units.size() * sizeof(Unit);
  const size_t n_tab = plan->host.tables.size() * sizeof(double);
  // Restore work items carry their page; only checkpoint plans read page tables on the device.
  const size_t n_pt = plan->host.kind == 1 ? plan->host.page_tables.size() * sizeof(int32_t) : 0;
  const size_t total = al(n_units) + al(n_tab) + al(n_pt);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) {
    delete plan;
    return PKV_ERR_DEVICE;
  }
  plan->device = dev;
  plan->host.info.device = dev;
  // Residency cap through LDS: each restore workgroup claims a share of the
  // compute unit's LDS (it needs only its table) so that no more than
  // restore_workgroups_per_cu() fit.
  int lds_cu = 0, lds_wg = 0;
  if (hipDeviceGetAttribute(&lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) == hipSuccess &&
      hipDeviceGetAttribute(&lds_wg, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess && lds_cu > 0) {
    const int64_t table = int64_t(kMaxHeadDim) * int64_t(sizeof(double));
    const int64_t n = restore_workgroups_per_cu(plan->host);
    const int64_t share = (int64_t(lds_cu) / n + int64_t(lds_cu) / (n + 1)) / 2;
    const int64_t dyn = std::min<int64_t>((share - table) & ~int64_t(255), int64_t(lds_wg) - table);
    plan->restore_lds = n < 16 / std::max(1, plan->host.workgroup / 64) && dyn > 0 ? uint32_t(dyn) : 0;
  } else {
    (void)hipGetLastError();
  }
  // Late start order up to kLateRounds rounds of resident workgroups: with
  // 8B-shaped rows (690 units per layer of an 8K-token suffix, 512 resident)
  // it measured faster up to 4 layers (5.4 rounds), warm and cold, and
  // slower cold from 6 layers (8 rounds) on.  Rows narrow enough for
  // workgroups under kWorkgroup threads take it at any depth: on the 32-layer
  // 8B-shaped workload's share of one KV head per GPU (one-wave workgroups of
  // two tokens per thread) it measured 102-112 us against 127-135 us, and
  // within 1% of the early order at two and four heads.
  int cus = 0;
  if (plan->host.workgroup < kWorkgroup)
    plan->restore_late_units = INT64_MAX;
  else if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0)
    plan->restore_late_units = kLateRounds * int64_t(cus) * restore_workgroups_per_cu(plan->host);
  else
    (void)hipGetLastError();
  if (total > 0) {
    hipError_t e = hipMalloc(&plan->device_mem, total);
    if (e != hipSuccess) {
      plan->device_mem = nullptr;
      delete plan;
      return e == hipErrorOutOfMemory ? PKV_ERR_OUT_OF_MEMORY : PKV_ERR_DEVICE;
    }
    char* p = static_cast<char*>(plan->device_mem);
    plan->d_units = reinterpret_cast<Unit*>(p);
    p += al(n_units);
    plan->d_tables = reinterpret_cast<double*>(p);
    p += al(n_tab);
    plan->d_page_tables = reinterpret_cast<int32_t*>(p);
    bool ok = true;
    if (n_units) ok = ok && hipMemcpy(plan->d_units, plan->host.units.data(), n_units, hipMemcpyHostToDevice) == hipSuccess;
    if (n_tab) ok = ok && hipMemcpy(plan->d_tables, plan->host.tables.data(), n_tab, hipMemcpyHostToDevice) == hipSuccess;
    if (n_pt)
      ok = ok && hipMemcpy(plan->d_page_tables, plan->host.page_tables.data(), n_pt, hipMemcpyHostToDevice) == hipSuccess;
    if (!ok) {
      (void)hipFree(plan->device_mem);
      delete plan;
      return PKV_ERR_DEVICE;
    }
  }
  // The device copy is authoritative; keep only the metadata on the host.
  std::vector<Unit>().swap(plan->host.units);
  std::vector<double>().swap(plan->host.tables);
  std::vector<int32_t>().swap(plan->host.page_tables);
  *out = plan;
  return PKV_OK;
}

// Where a kernel may read or write a buffer: device or managed memory of the
// plan's device as is; pinned host memory through its device mapping (the
// kernel then reaches it over the host link).  Pageable host memory, or
// memory of another device, is rejected: the kernel would fault on it.
pkv_status_t kernel_accessible(const pkv_plan* plan, const void* p, const void** out) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return PKV_ERR_INVALID_ARGUMENT;
  }
  if ((a.type == hipMemoryTypeDevice || a.type == hipMemoryTypeManaged) && a.device == plan->device) {
    *out = p;
    return PKV_OK;
  }
  if (a.type == hipMemoryTypeHost && a.devicePointer) {
    *out = a.devicePointer;
    return PKV_OK;
  }
  return PKV_ERR_INVALID_ARGUMENT;
}

// Caches must be device (or managed) memory of the plan's device.
pkv_status_t device_resident(const pkv_plan* plan, const void* p) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return PKV_ERR_INVALID_ARGUMENT;
  }
  return (a.type == hipMemoryTypeDevice || a.type == hipMemoryTypeManaged) && a.device == plan->device
             ? PKV_OK
             : PKV_ERR_INVALID_ARGUMENT;
}

// Pointer, alignment, size and overlap checks shared by both restore entry points.
pkv_status_t check_restore_buffers(const pkv_plan* plan, const void* payload, uint64_t payload_bytes,
                                   const void* scales, uint64_t scale_bytes, const void* k_cache, const void* v_cache,
                                   uint64_t cache_bytes) {
  const pkv_plan_info_t& info = plan->host.info;
  if (!payload || !scales || !k_cache || !v_cache) return PKV_ERR_INVALID_ARGUMENT;
  if (reinterpret_cast<uintptr_t>(payload) % 16 || reinterpret_cast<uintptr_t>(scales) % 8)
    return PKV_ERR_INVALID_ARGUMENT;
  if (payload_bytes < info.payload_bytes || scale_bytes < info.scale_bytes || cache_bytes < info.cache_bytes)
    return PKV_ERR_INVALID_ARGUMENT;
  ByteRange caches[2];
  int n = 0;
  if (!cache_ranges(plan->host.model, k_cache, v_cache, info.cache_bytes, caches, n)) return PKV_ERR_INVALID_ARGUMENT;
  for (int i = 0; i < n; ++i)
    if (ranges_overlap(caches[i].p, caches[i].n, payload, info.payload_bytes) ||
        ranges_overlap(caches[i].p, caches[i].n, scales, info.scale_bytes))
      return PKV_ERR_INVALID_ARGUMENT;
  return PKV_OK;
}

// Start order of the restore kernel: 0 by plan and launch size (late for
// narrow rows and for launches of at most kLateRounds rounds of resident
// workgroups), 1 early, 2 late.
// Set only through the test hook pkv_internal_set_restore_order.
std::atomic<int> g_restore_order{0};

// Enqueue the restore kernel over units [u0, u0 + n) of the plan, those whose
// K rows start in payload bytes [win_lo, win_hi).
pkv_status_t launch_restore(const pkv_plan* plan, const void* payload, const void* scales, void* k_cache,
                            void* v_cache, int64_t u0, int64_t n, hipStream_t stream, uint64_t win_lo = 0,
                            uint64_t win_hi = ~uint64_t(0)) {
  const pkv_model_t& m = plan->host.model;
  KernelArgs a;
  a.win_lo = win_lo;
  a.win_hi = win_hi;
  a.units = plan->d_units + u0;
  a.tables = plan->d_tables;
  a.payload = static_cast<const uint8_t*>(payload);
  a.scales = static_cast<const uint16_t*>(scales);
  a.k_cache = static_cast<uint16_t*>(k_cache);
  a.v_cache = static_cast<uint16_t*>(v_cache);
  a.layer_elems = layer_elems(m);
  a.page_shift = page_shift(m);
  a.H = m.num_kv_heads;
  a.D = m.head_dim;
  a.log2P = plan->host.log2_page;
  a.cols = m.num_kv_heads * m.head_dim / 16;
  a.tpp = plan->host.workgroup / a.cols;
  auto shift_of = [](int32_t x) {
    int32_t s = 0;
    while ((1 << s) < x) ++s;
    return (1 << s) == x ? s : -1;
  };
  a.cols_shift = shift_of(a.cols);
  a.dq_shift = shift_of(m.head_dim / 16);
  a.R = m.rotary_dim ? m.rotary_dim : m.head_dim;
  const dim3 grid(static_cast<uint32_t>(n)), block(plan->host.workgroup);
  const bool bf16 = m.out_dtype == PKV_OUT_BF16, half = m.rope_style == PKV_ROPE_HALF;
  const int order = g_restore_order.load(std::memory_order_relaxed);
  const bool late = order == 2 || (order == 0 && n <= plan->restore_late_units);
  const uint32_t lds = plan->restore_lds;
  if (late) {
    if (bf16 && half)
      hipLaunchKernelGGL((restore_kernel<true, PKV_ROPE_HALF, true>), grid, block, lds, stream, a);
    else if (bf16)
      hipLaunchKernelGGL((restore_kernel<true, PKV_ROPE_INTERLEAVED, true>), grid, block, lds, stream, a);
    else if (half)
      hipLaunchKernelGGL((restore_kernel<false, PKV_ROPE_HALF, true>), grid, block, lds, stream, a);
    else
      hipLaunchKernelGGL((restore_kernel<false, PKV_ROPE_INTERLEAVED, true>), grid, block, lds, stream, a);
  } else {
    if (bf16 && half)
      hipLaunchKernelGGL((restore_kernel<true, PKV_ROPE_HALF, false>), grid, block, lds, stream, a);
    else if (bf16)
      hipLaunchKernelGGL((restore_kernel<true, PKV_ROPE_INTERLEAVED, false>), grid, block, lds, stream, a);
    else if (half)
      hipLaunchKernelGGL((restore_kernel<false, PKV_ROPE_HALF, false>), grid, block, lds, stream, a);
    else
      hipLaunchKernelGGL((restore_kernel<false, PKV_ROPE_INTERLEAVED, false>), grid, block, lds, stream, a);
  }
  return hipGetLastError() == hipSuccess ? PKV_OK : PKV_ERR_DEVICE;
}

}  // namespace pkv

// Staging buffer of pkv_restore_from_host_noalloc: payload windows in the
// first kStagePayloadBytes, one request-layer's scales after them.  Each GPU
// the library runs on holds its own copy until the process ends.  In host
// code this name is not a device address: the entry point takes the address
// from hipGetSymbolAddress, once per device (stage_address).
static __device__ __align__(256) unsigned char scratch[pkv::kStagePayloadBytes + pkv::kStageScaleBytes];

namespace pkv {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_stage_mu;
void* g_stage[kMaxDevices] = {};

// Device address of `scratch` on device `dev` (the current device).
pkv_status_t stage_address(int dev, uint8_t** out) {
  if (dev < 0 || dev >= kMaxDevices) return PKV_ERR_DEVICE;
  std::lock_guard<std::mutex> lock(g_stage_mu);
  if (!g_stage[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return PKV_ERR_DEVICE;
    }
    g_stage[dev] = p;
  }
  *out = static_cast<uint8_t*>(g_stage[dev]);
  return PKV_OK;
}

// Pinned host memory only: asynchronous copies from it need no staging by
// the runtime.
bool pinned_host(const void* p) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return a.type == hipMemoryTypeHost;
}

}  // namespace
}  // namespace pkv

extern "C" {

// Internal test hook (not part of pkv.h): force the restore kernel's start
// order for every later launch in the process (0: by launch size, 1: early,
// 2: late), so that tests cover both orders on every shape.
pkv_status_t pkv_internal_set_restore_order(int32_t order) {
  if (order < 0 || order > 2) return PKV_ERR_INVALID_ARGUMENT;
  pkv::g_restore_order.store(order, std::memory_order_relaxed);
  return PKV_OK;
}

pkv_status_t pkv_restore_plan(const pkv_model_t* model, const pkv_request_t* requests, int32_t num_requests,
                              pkv_plan_t** out) {
  if (!out) return PKV_ERR_INVALID_ARGUMENT;
  *out = nullptr;
  pkv::HostPlan hp;
  const pkv_status_t st = pkv::build_host_plan(model, requests, num_requests, &hp);
  if (st != PKV_OK) return st;
  return pkv::upload_plan(std::move(hp), out);
}

pkv_status_t pkv_restore(const pkv_plan_t* plan, const void* payload, uint64_t payload_bytes, const void* scales,
                         uint64_t scale_bytes, void* k_cache, void* v_cache, uint64_t cache_bytes, void* hip_stream) {
  if (!plan || plan->host.kind != 0) return PKV_ERR_INVALID_ARGUMENT;
  const pkv_plan_info_t& info = plan->host.info;
  if (info.num_units == 0) return PKV_OK;
  pkv_status_t st = pkv::check_restore_buffers(plan, payload, payload_bytes, scales, scale_bytes, k_cache, v_cache,
                                              cache_bytes);
  if (st != PKV_OK) return st;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != plan->device) return PKV_ERR_DEVICE;
  const void *p_dev = nullptr, *s_dev = nullptr;
  if ((st = pkv::kernel_accessible(plan, payload, &p_dev)) != PKV_OK ||
      (st = pkv::kernel_accessible(plan, scales, &s_dev)) != PKV_OK || (st = pkv::device_resident(plan, k_cache)) != PKV_OK ||
      (st = pkv::device_resident(plan, v_cache)) != PKV_OK)
    return st;
  return pkv::launch_restore(plan, p_dev, s_dev, k_cache, v_cache, 0, info.num_units,
                             static_cast<hipStream_t>(hip_stream));
}

pkv_status_t pkv_restore_from_host(const pkv_plan_t* plan, const void* host_payload, uint64_t host_payload_bytes,
                                   const void* host_scales, uint64_t host_scale_bytes, void* payload,
                                   uint64_t payload_bytes, void* scales, uint64_t scale_bytes, void* k_cache,
                                   void* v_cache, uint64_t cache_bytes, void* hip_stream) {
  if (!plan || plan->host.kind != 0) return PKV_ERR_INVALID_ARGUMENT;
  const pkv_plan_info_t& info = plan->host.info;
  if (info.num_units == 0) return PKV_OK;
  pkv_status_t st = pkv::check_restore_buffers(plan, payload, payload_bytes, scales, scale_bytes, k_cache, v_cache,
                                              cache_bytes);
  if (st != PKV_OK) return st;
  if (!host_payload || !host_scales || host_payload_bytes < info.payload_bytes || host_scale_bytes < info.scale_bytes)
    return PKV_ERR_INVALID_ARGUMENT;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != plan->device) return PKV_ERR_DEVICE;
  if ((st = pkv::device_resident(plan, payload)) != PKV_OK || (st = pkv::device_resident(plan, scales)) != PKV_OK ||
      (st = pkv::device_resident(plan, k_cache)) != PKV_OK || (st = pkv::device_resident(plan, v_cache)) != PKV_OK)
    return st;
  pkv_plan* p = const_cast<pkv_plan*>(plan);  // the copy streams and events are created on first use
  const int64_t L = plan->host.model.num_layers;
  if (p->copy_streams.empty()) {  // all or nothing
    std::vector<void*> streams, events;
    bool ok = true;
    for (int i = 0; ok && i < pkv::kHostCopyStreams; ++i) {
      hipStream_t cs = nullptr;
      ok = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking) == hipSuccess;
      if (ok) streams.push_back(cs);
    }
    for (int64_t i = 0; ok && i < 1 + L * pkv::kHostCopyStreams; ++i) {
      hipEvent_t e = nullptr;
      ok = hipEventCreateWithFlags(&e, hipEventDisableTiming) == hipSuccess;
      if (ok) events.push_back(e);
    }
    if (!ok) {
      for (void* e : events) (void)hipEventDestroy(static_cast<hipEvent_t>(e));
      for (void* cs : streams) (void)hipStreamDestroy(static_cast<hipStream_t>(cs));
      return PKV_ERR_DEVICE;
    }
    p->copy_streams = std::move(streams);
    p->events = std::move(events);
  }
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  const size_t n_copy = p->copy_streams.size();
  auto ev = [&](int64_t i) { return static_cast<hipEvent_t>(p->events[size_t(i)]); };
  // Earlier work on the caller's stream may still read `payload`.
  if (hipEventRecord(ev(0), stream) != hipSuccess) return PKV_ERR_DEVICE;
  for (size_t i = 0; i < n_copy; ++i)
    if (hipStreamWaitEvent(static_cast<hipStream_t>(p->copy_streams[i]), ev(0), 0) != hipSuccess)
      return PKV_ERR_DEVICE;
  const uint8_t* hp_bytes = static_cast<const uint8_t*>(host_payload);
  const uint8_t* hs_bytes = static_cast<const uint8_t*>(host_scales);
  uint8_t* dp_bytes = static_cast<uint8_t*>(payload);
  uint8_t* ds_bytes = static_cast<uint8_t*>(scales);
  const pkv::HostPlan& h = plan->host;
  // Copies are cut into chunks of at most kHostChunkBytes and dealt to the
  // copy streams in turn, so every stream (each feeding its own DMA engine)
  // stays busy within a layer; layer l's restore waits on every stream that
  // carried one of its chunks.
  size_t next = 0;
  auto enqueue = [&](uint8_t* dst, const uint8_t* src, const pkv::CopyRange& c, uint32_t& used) {
    for (uint64_t o = 0; o < c.len; o += pkv::kHostChunkBytes) {
      const uint64_t n = c.len - o < pkv::kHostChunkBytes ? c.len - o : pkv::kHostChunkBytes;
      const size_t k = next++ % n_copy;
      if (hipMemcpyAsync(dst + c.off + o, src + c.off + o, n, hipMemcpyHostToDevice,
                         static_cast<hipStream_t>(p->copy_streams[k])) != hipSuccess)
        return false;
      used |= 1u << k;
    }
    return true;
  };
  for (int64_t l = 0; l < L; ++l) {
    uint32_t used = 0;
    for (int64_t i = h.payload_layer[l]; i < h.payload_layer[l + 1]; ++i)
      if (!enqueue(dp_bytes, hp_bytes, h.payload_ranges[size_t(i)], used)) return PKV_ERR_DEVICE;
    for (int64_t i = h.scale_layer[l]; i < h.scale_layer[l + 1]; ++i)
      if (!enqueue(ds_bytes, hs_bytes, h.scale_ranges[size_t(i)], used)) return PKV_ERR_DEVICE;
    for (size_t k = 0; k < n_copy; ++k) {
      if (!(used & (1u << k))) continue;
      hipEvent_t e = ev(1 + l * int64_t(n_copy) + int64_t(k));
      if (hipEventRecord(e, static_cast<hipStream_t>(p->copy_streams[k])) != hipSuccess ||
          hipStreamWaitEvent(stream, e, 0) != hipSuccess)
        return PKV_ERR_DEVICE;
    }
    const int64_t u0 = h.layer_units[l], n = h.layer_units[l + 1] - u0;
    if (n == 0) continue;
    st = pkv::launch_restore(plan, payload, scales, k_cache, v_cache, u0, n, stream);
    if (st != PKV_OK) return st;
  }
  return PKV_OK;
}

pkv_status_t pkv_restore_from_host_noalloc(const pkv_plan_t* plan, const void* host_payload,
                                           uint64_t host_payload_bytes, const void* host_scales,
                                           uint64_t host_scale_bytes, void* k_cache, void* v_cache,
                                           uint64_t cache_bytes, void* hip_stream) {
  if (!plan || plan->host.kind != 0) return PKV_ERR_INVALID_ARGUMENT;
  const pkv::HostPlan& h = plan->host;
  const pkv_plan_info_t& info = h.info;
  if (info.num_units == 0) return PKV_OK;
  if (!host_payload || !host_scales || !k_cache || !v_cache) return PKV_ERR_INVALID_ARGUMENT;
  if (host_payload_bytes < info.payload_bytes || host_scale_bytes < info.scale_bytes || cache_bytes < info.cache_bytes)
    return PKV_ERR_INVALID_ARGUMENT;
  pkv::ByteRange caches[2];
  int n_caches = 0;
  if (!pkv::cache_ranges(h.model, k_cache, v_cache, info.cache_bytes, caches, n_caches)) return PKV_ERR_INVALID_ARGUMENT;
  // Size limit: one request-layer's scales must fit the scale stage.
  if (!h.stage_ok) return PKV_ERR_INVALID_ARGUMENT;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != plan->device) return PKV_ERR_DEVICE;
  if (!pkv::pinned_host(host_payload) || !pkv::pinned_host(host_scales)) return PKV_ERR_INVALID_ARGUMENT;
  pkv_status_t st;
  if ((st = pkv::device_resident(plan, k_cache)) != PKV_OK || (st = pkv::device_resident(plan, v_cache)) != PKV_OK)
    return st;
  uint8_t* stage = nullptr;
  if ((st = pkv::stage_address(dev, &stage)) != PKV_OK) return st;
  uint8_t* stage_scales = stage + pkv::kStagePayloadBytes;
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  const uint8_t* hp = static_cast<const uint8_t*>(host_payload);
  const uint8_t* hs = static_cast<const uint8_t*>(host_scales);
  // Every step goes on the caller's stream, so a step's copies wait for the
  // restore of the step before it, which still reads the stage.
  for (const pkv::StageStep& step : h.stage_steps) {
    if (step.scale_elems &&
        hipMemcpyAsync(stage_scales, hs + step.scale0 * 2, step.scale_elems * 2, hipMemcpyHostToDevice, stream) !=
            hipSuccess)
      return PKV_ERR_DEVICE;
    for (int64_t c = step.copy0; c < step.copy1; ++c) {
      const pkv::StageCopy& cp = h.stage_copies[size_t(c)];
      if (hipMemcpyAsync(stage + cp.dst, hp + cp.src, cp.len, hipMemcpyHostToDevice, stream) != hipSuccess)
        return PKV_ERR_DEVICE;
    }
    // The kernel adds a unit's absolute checkpoint offsets to these bases:
    // payload byte o of the window is stage byte o - win_lo, scale element e
    // of the request-layer is stage element e - scale0.
    const void* payload_base = reinterpret_cast<const void*>(reinterpret_cast<uintptr_t>(stage) - step.win_lo);
    const void* scales_base =
        reinterpret_cast<const void*>(reinterpret_cast<uintptr_t>(stage_scales) - step.scale0 * 2);
    st = pkv::launch_restore(plan, payload_base, scales_base, k_cache, v_cache, step.u0, step.u1 - step.u0, stream,
                             step.win_lo, step.win_hi);
    if (st != PKV_OK) return st;
  }
  return PKV_OK;
}

void pkv_free(pkv_plan_t* plan) {
  if (!plan) return;
  if (plan->device_mem || !plan->copy_streams.empty()) {
    int cur = -1;
    const bool switched = hipGetDevice(&cur) == hipSuccess && cur != plan->device &&
                          hipSetDevice(plan->device) == hipSuccess;
    for (void* e : plan->events)
      if (e) (void)hipEventDestroy(static_cast<hipEvent_t>(e));
    for (void* cs : plan->copy_streams) (void)hipStreamDestroy(static_cast<hipStream_t>(cs));
    if (plan->device_mem) (void)hipFree(plan->device_mem);
    if (switched) (void)hipSetDevice(cur);
  }
  delete plan;
}

pkv_status_t pkv_plan_payload_bytes(const pkv_plan_t* plan, int32_t req, uint64_t* bytes) {
  if (!plan || !bytes || req < 0 || size_t(req) >= plan->host.req_payload_bytes.size()) return PKV_ERR_INVALID_ARGUMENT;
  *bytes = plan->host.req_payload_bytes[size_t(req)];
  return PKV_OK;
}

pkv_status_t pkv_plan_query(const pkv_plan_t* plan, pkv_plan_info_t* info) {
  if (!plan || !info) return PKV_ERR_INVALID_ARGUMENT;
  *info = plan->host.info;
  return PKV_OK;
}

}  // extern "C"
