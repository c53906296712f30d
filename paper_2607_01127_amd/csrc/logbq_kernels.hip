// gfx950 kernels of liblogbq and the device entry points of the C ABI.
//
//   k_encode   Quant (Eq. 1): float32 weights -> packed sign+magnitude nibbles, by comparing
//              |x| with the exact per-tensor thresholds (7 compares per weight).
//   k_dequant  Dequant (Eq. 2) by codebook lookup: nibbles -> float32 (bit-exact).
//   k_gemv     y = x . W_hat^T for m <= 8 batch rows: packed codes stream from HBM with 128-bit
//              non-temporal loads; each code byte (two weights) indexes a 256-entry table of
//              float16 pairs held in LDS (one private copy per lane, so lookups never conflict on
//              a bank); v_dot2_f32_f16 accumulates in float32; DPP row reductions plus lane reads
//              finish the wavefront sum.
//   k_mfma2    y = x . W_hat^T for larger m: a code dword (8 weights of one row) becomes one
//              lane's B operand of v_mfma_f32_16x16x32_f16, dequantized by pair-table lookups
//              or by v_perm_b32 byte tables in registers; activations are staged through LDS
//              as the A operand; float32 accumulation in the MFMA. k_mfma2_narrow: the same
//              with 64-row workgroups, for layers whose workgroups then all fit on the chip.
//   k_mfma_sk  the same product for 2 <= m <= 32 split over K: the 8 or 16 wavefronts of a
//              workgroup share a block of 16 rows (one K slice each, activations held in
//              registers) and sum their partial tiles through LDS; at K = 8192 and m > 16, on
//              narrow layers, and at K = 14336, two workgroups share a block (one K half each)
//              and add into a zeroed y.
//   k_mfma_sk8 the split-K product on 8-bit codes (m <= 16), weights looked up in an LDS table.
//   k_mfma_kq  the same product for m > 96: each wavefront takes 64 weight rows and one K
//              quarter of every step for all 128 batch rows of the workgroup; the quarters'
//              tiles are summed through LDS at the end (k_mfma_kq8: the same on 8-bit codes).
//   k_encode8, k_dequant8, k_gemv<8, ...>, k_mfma2<8, ...>  the same on 8-bit codes.
//   k_encode_uniform  codes of the asymmetric linear baseline (Sec. 2), for comparisons.
//   k_gptq_panel, k_gptq_trail  GPTQ calibration with a fixed codebook (one wavefront per row
//              within a block of 128 columns; the block's errors applied to the later columns).
//   k_fit_hist  the device fit's radix-selection passes (Eq. 5 with exact sums): per-bin counts
//              and exact integer energy sums of |w| binned by its float32 bit pattern.
//
// The float16 tables hold codebook / 2^e with 2^e chosen so that the largest entry lies in
// [2^14, 2^15); the result is multiplied back by 2^e (exact). Lookup replaces evaluating
// b^(|q| - s) per weight, as in Sec. 3.3 of the paper.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <vector>

#include "fit_detail.h"
#include "logbq.h"

namespace {

typedef _Float16 half_t;
typedef half_t half2v __attribute__((ext_vector_type(2)));
typedef half_t half8v __attribute__((ext_vector_type(8)));
typedef float float16v __attribute__((ext_vector_type(16)));
typedef float float4v __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
// Pointers into global memory, so that loads through them are global (not flat) loads.
typedef const __attribute__((address_space(1))) uint8_t* GlobalU8;
typedef const __attribute__((address_space(1))) u32x4* GlobalU32x4;

// Word 3 of a gfx9 buffer resource descriptor for untyped (raw) 32-bit access.
constexpr int kBufferRsrcWord3 = 0x00020000;
// Cache policy bits of a buffer load: non-temporal (streamed once).
constexpr int kCachePolicyNT = 2;

struct Thresholds { float t[7]; };
// 8-bit thresholds plus the log-domain estimate of a magnitude index: index ~ floor(log2|x| *
// inv + c), inv = 1 / log2 b, c = s + 1/2 (inv = 0: no estimate, binary search only).
struct Thresholds8 { float t[127]; float inv, c; };
struct Codebook32 { float v[16]; };
struct Lut16 { uint32_t h[8]; };     // h[i] = f16(lut[2i]) | f16(lut[2i+1]) << 16
struct Lut256 { uint32_t h[128]; };  // the same for the 256 entries of an 8-bit codebook
template <int BITS> struct LutOf;
template <> struct LutOf<4> { using type = Lut16; };
template <> struct LutOf<8> { using type = Lut256; };

constexpr int kLutEntries = 256;   // one entry per code byte (two nibbles)
constexpr int kLutCopies = 64;     // one copy per lane of a wavefront
constexpr int kLutWords = kLutEntries * kLutCopies;

// ------------------------------------------------------------------ encode
// A wavefront encodes tiles of 64 * U float4 chunks (4 weights -> one 16-bit code group):
// load j of lane l reads chunk tile * 64U + 64 j + l, so every load instruction covers 1 KiB of
// contiguous weights and every store 128 contiguous bytes of codes; U loads are in flight per
// lane. Chunk indices past the end are clamped for loading and not stored.
constexpr int kEncU = 8;

__device__ __forceinline__ uint32_t encode4(const f32x4 a, const Thresholds& th) {
  const float v[4] = {a.x, a.y, a.z, a.w};
  uint32_t out = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float x = v[j];
    const float ax = __builtin_fabsf(x);
    uint32_t mag = 0;
#pragma unroll
    for (int t = 0; t < 7; ++t) mag += (ax >= th.t[t]) ? 1u : 0u;
    const uint32_t sgn = (x < 0.0f && mag != 0u) ? 8u : 0u;
    out |= (mag | sgn) << (4 * j);
  }
  return out;
}

// Asymmetric linear baseline (Sec. 2): the unsigned 4-bit code of x is the number of the 15
// non-decreasing thresholds at or below it.
struct ThresholdsU { float t[15]; };

__device__ __forceinline__ uint32_t encode4(const f32x4 a, const ThresholdsU& th) {
  const float v[4] = {a.x, a.y, a.z, a.w};
  uint32_t out = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint32_t q = 0;
#pragma unroll
    for (int t = 0; t < 15; ++t) q += (v[j] >= th.t[t]) ? 1u : 0u;
    out |= q << (4 * j);
  }
  return out;
}

template <typename TH>
__device__ __forceinline__ void encode_tiles(const f32x4* __restrict__ w,
                                             uint16_t* __restrict__ codes, int64_t nchunk,
                                             const TH& th) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 6;   // 256-thread blocks
  const int64_t nwaves = ((int64_t)gridDim.x * 256) >> 6;
  const int64_t ntiles = (nchunk + 64 * kEncU - 1) / (64 * kEncU);
  for (int64_t t = wave; t < ntiles; t += nwaves) {
    const int64_t base = t * 64 * kEncU + lane;
    f32x4 v[kEncU];
#pragma unroll
    for (int j = 0; j < kEncU; ++j) {
      const int64_t idx = base + 64 * j;
      v[j] = __builtin_nontemporal_load(w + (idx < nchunk ? idx : nchunk - 1));
    }
#pragma unroll
    for (int j = 0; j < kEncU; ++j) {
      const int64_t idx = base + 64 * j;
      if (idx < nchunk) codes[idx] = (uint16_t)encode4(v[j], th);
    }
  }
}

__global__ __launch_bounds__(256) void k_encode(const f32x4* __restrict__ w,
                                                uint16_t* __restrict__ codes, int64_t nchunk,
                                                Thresholds th) {
  encode_tiles(w, codes, nchunk, th);
}

__global__ __launch_bounds__(256) void k_encode_uniform(const f32x4* __restrict__ w,
                                                        uint16_t* __restrict__ codes,
                                                        int64_t nchunk, ThresholdsU th) {
  encode_tiles(w, codes, nchunk, th);
}

// ------------------------------------------------------------------ dequantize
__global__ __launch_bounds__(256) void k_dequant(const uint32_t* __restrict__ codes,
                                                 f32x4* __restrict__ w, int64_t nwords,
                                                 Codebook32 cb) {
  __shared__ float s_cb[16];
  if (threadIdx.x < 16) s_cb[threadIdx.x] = cb.v[threadIdx.x];
  __syncthreads();
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nwords; i += stride) {
    const uint32_t c = codes[i];
    f32x4 a, b;
    a.x = s_cb[c & 15u];         a.y = s_cb[(c >> 4) & 15u];
    a.z = s_cb[(c >> 8) & 15u];  a.w = s_cb[(c >> 12) & 15u];
    b.x = s_cb[(c >> 16) & 15u]; b.y = s_cb[(c >> 20) & 15u];
    b.z = s_cb[(c >> 24) & 15u]; b.w = s_cb[c >> 28];
    __builtin_nontemporal_store(a, w + 2 * i);
    __builtin_nontemporal_store(b, w + 2 * i + 1);
  }
}

// 8-bit codes. Encode: the magnitude index of |x| is the number of the 127 sorted thresholds at
// or below it. Threshold k sits at b^(k + 1/2 - s) (Eq. 1's rounding in the log domain), so
// floor(log2|x| / log2 b + s + 1/2) is the index up to one step near a threshold; comparing
// |x| with the thresholds on both sides of that estimate (a copy in LDS) makes it exact. The
// host checks that every threshold lies within a quarter step of where the estimate puts it
// and that b is not so close to 1 that float rounding of the estimate exceeds a tenth of a
// step, which bounds the estimate's error by one step; otherwise (and for zero, subnormal, infinite
// or NaN |x|) a 7-step binary search over the thresholds decides. Measured on MI355X (the
// 8192 x 28672 tensor): 228.5 -> 209.8 us with the grid at 64 workgroups per CU. One code
// byte per weight, four per float4 chunk (stored as one dword). Tiles as in k_encode.
__global__ __launch_bounds__(256) void k_encode8(const f32x4* __restrict__ w,
                                                 uint32_t* __restrict__ codes, int64_t nchunk,
                                                 Thresholds8 th) {
  __shared__ float s_t[128];
  if (threadIdx.x < 127) s_t[threadIdx.x] = th.t[threadIdx.x];
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  const int64_t ntiles = (nchunk + 64 * kEncU - 1) / (64 * kEncU);
  for (int64_t t = wave; t < ntiles; t += nwaves) {
    const int64_t base = t * 64 * kEncU + lane;
    f32x4 v[kEncU];
#pragma unroll
    for (int j = 0; j < kEncU; ++j) {
      const int64_t idx = base + 64 * j;
      v[j] = __builtin_nontemporal_load(w + (idx < nchunk ? idx : nchunk - 1));
    }
#pragma unroll
    for (int j = 0; j < kEncU; ++j) {
      const int64_t idx = base + 64 * j;
      const float e[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
      uint32_t out = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float ax = __builtin_fabsf(e[q]);
        uint32_t lo;   // the number of thresholds <= ax
        if (th.inv > 0.0f && ax >= 1.17549435e-38f && ax <= 3.40282347e38f) {
          const float f = __builtin_amdgcn_logf(ax) * th.inv + th.c;   // log2
          int est = (int)__builtin_floorf(f);
          est = est < 0 ? 0 : (est > 127 ? 127 : est);
          if (est < 127 && s_t[est] <= ax) ++est;
          if (est > 0 && s_t[est - 1] > ax) --est;
          lo = (uint32_t)est;
        } else {
          lo = 0;   // thresholds s_t[0 .. lo) are <= ax; the steps sum to 127
#pragma unroll
          for (int step = 64; step >= 1; step >>= 1)
            if (s_t[lo + step - 1] <= ax) lo += step;
        }
        const uint32_t sgn = (e[q] < 0.0f && lo != 0u) ? 128u : 0u;
        out |= (lo | sgn) << (8 * q);
      }
      if (idx < nchunk) codes[idx] = out;
    }
  }
}

struct Codebook256 { float v[256]; };

// Dequantize 8-bit codes: four codes per thread and step, one 16-byte store.
__global__ __launch_bounds__(256) void k_dequant8(const uint32_t* __restrict__ codes,
                                                  f32x4* __restrict__ w, int64_t nwords,
                                                  Codebook256 cb) {
  __shared__ float s_cb[256];
  s_cb[threadIdx.x] = cb.v[threadIdx.x];
  __syncthreads();
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nwords; i += stride) {
    const uint32_t c = codes[i];
    f32x4 a;
    a.x = s_cb[c & 255u]; a.y = s_cb[(c >> 8) & 255u];
    a.z = s_cb[(c >> 16) & 255u]; a.w = s_cb[c >> 24];
    __builtin_nontemporal_store(a, w + i);
  }
}

// y[0 .. count) = 0 with 16-byte stores (y is 16-byte aligned); the count % 4 floats of the
// tail are written by the first threads.
__global__ __launch_bounds__(256) void k_fill_zero(float* __restrict__ y, int64_t count) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t n4 = count >> 2;
  f32x4* y4 = reinterpret_cast<f32x4*>(y);
  for (int64_t i = t0; i < n4; i += stride) y4[i] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  if (t0 < (count & 3)) y[(n4 << 2) + t0] = 0.0f;
}

// ------------------------------------------------------------------ shared device helpers

// float16 bits of table entry c (0..15).
__device__ __forceinline__ uint32_t lut16_entry(const Lut16 lut, uint32_t c) {
  const uint32_t i = c >> 1;
  uint32_t w = lut.h[0];
  w = (i == 1) ? lut.h[1] : w; w = (i == 2) ? lut.h[2] : w; w = (i == 3) ? lut.h[3] : w;
  w = (i == 4) ? lut.h[4] : w; w = (i == 5) ? lut.h[5] : w; w = (i == 6) ? lut.h[6] : w;
  w = (i == 7) ? lut.h[7] : w;
  return (c & 1u) ? (w >> 16) : (w & 0xFFFFu);
}

// Fill the LDS pair table: word (e * 64 + lane) = f16(lut[e & 15]) | f16(lut[e >> 4]) << 16,
// i.e. the two weights of code byte e in k order (low nibble = even k). Thread t writes the
// 16-byte vectors t + THREADS * i, so each store instruction covers contiguous LDS and never
// conflicts on a bank; vector v holds entry v / 16. With THREADS a multiple of 256, the low
// nibble of every entry a thread writes is the same, (t / 16) % 16, and the high nibbles are
// t / 256 + (THREADS / 256) * i: one select chain plus one halfword pick per vector.
template <int THREADS>
__device__ __forceinline__ void fill_pair_lut(uint32_t* s_lut, const Lut16 lut) {
  static_assert(THREADS % 256 == 0, "the low nibble must be fixed per thread");
  constexpr int kVecs = kLutWords / 4;
  const int t = threadIdx.x;
  const uint32_t lo = lut16_entry(lut, ((uint32_t)t >> 4) & 15u);
#pragma unroll
  for (int i = 0; i < kVecs / THREADS; ++i) {
    const uint32_t hn = ((uint32_t)t >> 8) + (uint32_t)(THREADS / 256) * (uint32_t)i;
    uint32_t hi;
    if (THREADS == 512) {
      // hn = (t >> 8) + 2 i: entry 2 i + (t >> 8) is a half of pair word h[i]
      hi = (t & 256) ? (lut.h[i] >> 16) : (lut.h[i] & 0xFFFFu);
    } else {
      hi = lut16_entry(lut, hn);
    }
    const u32x4 vv = lo | (hi << 16);
    *reinterpret_cast<u32x4*>(s_lut + 4 * (t + THREADS * i)) = vv;
  }
}

// The float16 pair for byte `i` (0..3) of code dword `d`, read from this lane's private copy.
// v_perm_b32 builds the byte address (byte << 8) | (lane << 2) in one instruction.
__device__ __forceinline__ uint32_t pair_lookup(const uint32_t* s_lut, uint32_t d,
                                                uint32_t laneoff, int i) {
  const uint32_t sel = 0x0C0C0000u | ((uint32_t)(4 + i) << 8);
  const uint32_t addr = __builtin_amdgcn_perm(d, laneoff, sel);
  return *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(s_lut) + addr);
}

__device__ __forceinline__ half2v as_half2(uint32_t u) { return __builtin_bit_cast(half2v, u); }

// 8-bit codes: LDS word (e * 64 + lane) = f16(lut[e]) in its low half, one private copy per
// lane as for the pair table. Vector v of the fill holds entry v / 16; entry e is half e % 2
// of lut.h[e / 2]. For thread t = 64 w + l, e / 2 = 2 w + l / 32 + (THREADS / 32) i takes two
// values per wavefront, both read with uniform (scalar) loads of the kernel arguments: a load
// with a per-lane index would be a vector load that waits behind the code loads in flight.
template <int THREADS>
__device__ __forceinline__ void fill_single_lut(uint32_t* s_lut, const Lut256& lut) {
  constexpr int kVecs = kLutWords / 4;
  const int t = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const bool upper = (t & 32) != 0;
  const bool hi_half = (t & 16) != 0;
#pragma unroll
  for (int i = 0; i < kVecs / THREADS; ++i) {
    const int j = 2 * w + (THREADS / 32) * i;      // uniform
    const uint32_t h0 = lut.h[j], h1 = lut.h[j + 1];
    const uint32_t word = upper ? h1 : h0;
    const u32x4 vv = hi_half ? (word >> 16) : (word & 0xFFFFu);
    *reinterpret_cast<u32x4*>(s_lut + 4 * (t + THREADS * i)) = vv;
  }
}

template <int BITS, int THREADS>
__device__ __forceinline__ void fill_lut(uint32_t* s_lut, const typename LutOf<BITS>::type& lut) {
  if constexpr (BITS == 4) fill_pair_lut<THREADS>(s_lut, lut);
  else fill_single_lut<THREADS>(s_lut, lut);
}

// The float16 pair of 8-bit codes at bytes 2p and 2p + 1 (p = 0, 1) of code dword `d`.
__device__ __forceinline__ uint32_t single_pair(const uint32_t* s_lut, uint32_t d,
                                                uint32_t laneoff, int p) {
  const char* base = reinterpret_cast<const char*>(s_lut);
  const uint32_t a0 = __builtin_amdgcn_perm(d, laneoff, 0x0C0C0000u | ((uint32_t)(4 + 2 * p) << 8));
  const uint32_t a1 = __builtin_amdgcn_perm(d, laneoff, 0x0C0C0000u | ((uint32_t)(5 + 2 * p) << 8));
  const uint32_t lo = *reinterpret_cast<const uint16_t*>(base + a0);
  const uint32_t hi = *reinterpret_cast<const uint16_t*>(base + a1);
  return lo | (hi << 16);
}

template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
      0, __builtin_bit_cast(int, v), CTRL, ROW_MASK, 0xF, false));
}

// Sum over the 64 lanes of a wavefront; the result is valid in every lane.
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<0xB1>(v);    // quad_perm [1,0,3,2]
  v += dpp_f<0x4E>(v);    // quad_perm [2,3,0,1]
  v += dpp_f<0x124>(v);   // row_ror:4
  v += dpp_f<0x128>(v);   // row_ror:8   -> every lane holds its 16-lane row sum
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return (r0 + r1) + (r2 + r3);
}

// ------------------------------------------------------------------ GEMV, m <= 8
//
// One launch computes up to kMaxSegs linears that share the activations x (e.g. the query,
// key and value projections of a layer): segment s owns workgroups [wg_begin, next wg_begin)
// and its own codes, codebook table and output.
//
// Work split inside a segment: a workgroup of 8 wavefronts holds one LDS pair table. WK
// wavefronts share a row (each takes an interleaved slice of the row's 16-byte chunks). Lane `l`
// of wavefront `kw` in a group handles chunks c = s * 64 * WK + kw * 64 + l for s < CPL; its
// activations for those chunks (M rows x 32 values each) stay in registers for the whole kernel.
//
// Codes are read with buffer loads through a resource descriptor built per row in scalar
// registers (base = the row, size = its byte length); a row index past the end of the segment
// gets size 0, so its loads return zeros without touching memory. Chunk indices past the end of
// a row are clamped into it and meet zero activations.
//
// Rows, WK = 1: workgroup g (counted from the segment's first) owns the rows
// 8 g + t % 8 + (t / 8) * 8 G of its segment (G = the segment's workgroups), numbered by
// tickets t = 0, 1, ... in that order, so at any moment the chip streams one band of about 8 G
// consecutive rows. Wavefront w starts with tickets w, w + 8, ..., w + 8 (NBUF - 1) and takes
// every further ticket from an LDS counter as it finishes a row: the eight wavefronts of a CU
// share its rows dynamically and finish together (measured on MI355X: with fixed rows the
// wavefronts of one CU finished 1.5 to 2 us apart). Results stay in lanes (lane i holds the
// wavefront's i-th row) and are written 64 rows at a time, so no store waits among the code
// loads of the row loop.
// Rows, WK > 1: the 8 / WK groups of a workgroup take rows round-robin with the other groups
// of the segment, and reduce each row through LDS.
//
// Start-up: x (when M * K * 2 <= 32 KiB) is requested first and staged once per workgroup
// through LDS into registers; the first row of codes is requested next; the pair table is
// written while both are in flight; the rest of the ring follows. The row loop keeps NBUF code buffers: while one row is
// looked up, multiplied and reduced, the other NBUF - 1 are in flight. Every path through the
// loop issues the same loads, so the compiler waits for exactly the buffer it is about to use.
// NBUF is 3 when a row slice is at most two chunks per lane (and m <= 2) and 2 otherwise:
// measured on MI355X, about 4 to 8 KiB of codes in flight per wavefront streams best.
constexpr int kMaxSegs = 4;
constexpr int kStageXBytes = 32768;   // activations staged through LDS when M * K * 2 fits
// Staged activations keep every 64-byte chunk (the 32 values one lane multiplies with one
// 16-byte code chunk) at an 80-byte stride, so the four 16-byte reads of consecutive lanes
// fall on distinct LDS banks.
constexpr int kStageXPadded = kStageXBytes / 64 * 80;

template <int BITS>
struct GemvSeg {
  const uint8_t* codes;
  float* y;
  int n_rows;
  int wg_begin;
  int iters;
  float scale;
  typename LutOf<BITS>::type lut;
};
template <int BITS>
struct GemvSegs {
  GemvSeg<BITS> s[kMaxSegs];
  int count;
};

// Weights per 16-byte code chunk and activation dwords (float16 pairs) per chunk.
template <int BITS> constexpr int kChunkW = 128 / BITS;
template <int BITS> constexpr int kChunkX = 64 / BITS;

template <int BITS, int M, int CPL>
__device__ __forceinline__ void gemv_row(const u32x4 (&q)[CPL],
                                         const uint32_t (&xr)[M][CPL][kChunkX<BITS>],
                                         const uint32_t* s_lut, uint32_t laneoff,
                                         float (&acc)[M]) {
  float acc2[M];
#pragma unroll
  for (int m = 0; m < M; ++m) { acc[m] = 0.0f; acc2[m] = 0.0f; }
#pragma unroll
  for (int s = 0; s < CPL; ++s) {
    const uint32_t dw[4] = {q[s].x, q[s].y, q[s].z, q[s].w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      constexpr int P = BITS == 4 ? 4 : 2;   // float16 pairs per code dword
#pragma unroll
      for (int i = 0; i < P; ++i) {
        const half2v wp = as_half2(BITS == 4 ? pair_lookup(s_lut, dw[j], laneoff, i)
                                             : single_pair(s_lut, dw[j], laneoff, i));
#pragma unroll
        for (int m = 0; m < M; ++m) {
          float& a = (i & 1) ? acc2[m] : acc[m];
          a = __builtin_amdgcn_fdot2(wp, as_half2(xr[m][s][P * j + i]), a, false);
        }
      }
    }
  }
#pragma unroll
  for (int m = 0; m < M; ++m) acc[m] += acc2[m];
}

template <int BITS, int M, int CPL, bool SPLITK, int NBUF>
__global__ __launch_bounds__(512) void k_gemv(const uint16_t* __restrict__ x,
                                              const uint8_t* codes0, int k_cols, int n_rows0,
                                              int nseg, int wk_arg, int stage_x,
                                              GemvSegs<BITS> segs) {
  constexpr int CW = kChunkW<BITS>;   // weights per 16-byte code chunk
  constexpr int CX = kChunkX<BITS>;   // activation dwords per chunk
  const int wk = SPLITK ? wk_arg : 1;
  __shared__ __attribute__((aligned(16))) uint32_t s_lut[kLutWords];
  __shared__ __attribute__((aligned(16))) uint32_t s_x[kStageXPadded / 4];
  // Split rows: partial sums of kRed rows per wavefront, in two sets (see the loop below).
  constexpr int kRed = M <= 4 ? 16 : 8;
  __shared__ float s_part[SPLITK ? 2 : 1][SPLITK ? kRed : 1][8][M];
  __shared__ uint32_t s_ticket;

  // Segment of this workgroup: a uniform index, so its fields are scalar kernel-argument loads.
  // The first segment's codes pointer and row count (and the segment count) also come as
  // leading scalar arguments, which the hardware preloads into SGPRs: a one-segment launch
  // issues its first code loads without waiting for the segment table.
  const int bid = blockIdx.x;
  int si = 0;
  const uint8_t* codes = codes0;
  int n_rows = n_rows0;
  int wg_begin = 0;
  int next_begin = (int)gridDim.x;
  if (nseg > 1) {
    // A real branch (the empty asm keeps it from being turned into loads and selects that
    // would make the one-segment path wait for the table as well).
    asm volatile("" ::: "memory");
#pragma unroll
    for (int i = 1; i < kMaxSegs; ++i)
      if (i < nseg && bid >= segs.s[i].wg_begin) si = i;
    codes = segs.s[si].codes;
    n_rows = segs.s[si].n_rows;
    wg_begin = segs.s[si].wg_begin;
    next_begin = (si + 1 < nseg) ? segs.s[si + 1].wg_begin : (int)gridDim.x;
  }
  float* __restrict__ y = segs.s[si].y;
  const int iters = segs.s[si].iters;
  const float scale = segs.s[si].scale;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int kw = wave % wk;
  const int grp = wave / wk;
  const int groups = 8 / wk;
  const int nchunks = k_cols / CW;
  const int64_t row_bytes = (int64_t)k_cols * BITS / 8;
  const int total_groups = (next_begin - wg_begin) * groups;
  const int gid = (bid - wg_begin) * groups + grp;
  const uint32_t laneoff = (uint32_t)lane << 2;

  int coff[CPL];   // byte offset of this lane's chunk s within a row (clamped into the row)
  bool cval[CPL];
#pragma unroll
  for (int s = 0; s < CPL; ++s) {
    const int c = s * 64 * wk + kw * 64 + lane;
    cval[s] = c < nchunks;
    coff[s] = (cval[s] ? c : nchunks - 1) * 16;
  }

  auto load_row = [&](int r, u32x4 (&q)[CPL]) {
    const bool live = r < n_rows;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(codes + (live ? (int64_t)r * row_bytes : 0)), (short)0,
        live ? (int)row_bytes : 0, kBufferRsrcWord3);
#pragma unroll
    for (int s = 0; s < CPL; ++s)
      q[s] = __builtin_amdgcn_raw_buffer_load_b128(rs, coff[s], 0, kCachePolicyNT);
  };
  // Row of ticket t of this workgroup (WK = 1).
  const int wg_row0 = (bid - wg_begin) * 8;
  auto ticket_row = [&](uint32_t t) {
    return wg_row0 + (int)(t & 7u) + (int)(t >> 3) * total_groups;
  };

  u32x4 q[NBUF][CPL];
  int rq[NBUF];   // row held (or awaited) by buffer b; n_rows when none

  // Start-up, ordered so that the memory system is busy from the first cycle: the activations
  // are requested first (they return first), then the first row of codes; the pair table is
  // written while both are in flight. x is staged through LDS when it fits (M * K * 2 <= 32 KiB),
  // except for one batch row of one chunk per lane (K <= 2048), where each lane loads its 64
  // bytes straight into registers (measured on MI355X: 0.1-0.3 us faster per launch at
  // K = 2048, slower at K = 4096). Split rows that do not stage read x directly after the pair
  // table is written, which keeps their register use low.
  constexpr int kXVec = kStageXBytes / 16 / 512;     // 16-byte x vectors per thread
  u32x4 xv[kXVec];
  const int nvec = (M * k_cols) >> 3;                // 16-byte vectors of x
  const bool staged = stage_x != 0;
  if (staged) {
#pragma unroll
    for (int v = 0; v < kXVec; ++v) {
      const int i = threadIdx.x + 512 * v;
      xv[v] = *reinterpret_cast<const u32x4*>(x + 8 * (int64_t)(i < nvec ? i : 0));
    }
  }
  uint32_t xr[M][CPL][CX];
  // Unstaged activations of one-wavefront rows go out first, straight into registers.
  auto direct_x = [&]() {
#pragma unroll
    for (int s = 0; s < CPL; ++s) {
      const int c = s * 64 * wk + kw * 64 + lane;
#pragma unroll
      for (int m = 0; m < M; ++m)
#pragma unroll
        for (int qi = 0; qi < CX / 4; ++qi) {
          u32x4 v = 0;
          if (cval[s]) v = *reinterpret_cast<const u32x4*>(x + (int64_t)m * k_cols + (int64_t)c * CW + 8 * qi);
          xr[m][s][4 * qi] = v.x; xr[m][s][4 * qi + 1] = v.y;
          xr[m][s][4 * qi + 2] = v.z; xr[m][s][4 * qi + 3] = v.w;
        }
    }
  };
  if (!SPLITK && !staged) direct_x();
  // The first row goes out at once; the other NBUF - 1 rows right after the pair table is
  // written when the ring is three deep, after the barrier below when it is two deep (measured
  // on MI355X: issuing every ring row at once makes the first row arrive later, so with one or
  // two rows per wavefront both rows are computed after the last bytes land).
  constexpr bool kRestAfterFill = NBUF >= 3;
  if constexpr (!SPLITK) {
#pragma unroll
    for (int b = 0; b < NBUF; ++b) rq[b] = ticket_row((uint32_t)(wave + 8 * b));
    load_row(rq[0], q[0]);
    if (threadIdx.x == 0) s_ticket = 8 * NBUF;
  } else {
    load_row(gid, q[0]);
  }
  fill_lut<BITS, 512>(s_lut, segs.s[si].lut);
  if constexpr (!SPLITK && kRestAfterFill) {
#pragma unroll
    for (int b = 1; b < NBUF; ++b) load_row(rq[b], q[b]);
  }

  if (staged) {
#pragma unroll
    for (int v = 0; v < kXVec; ++v) {
      const int i = threadIdx.x + 512 * v;
      if (i < nvec) *reinterpret_cast<u32x4*>(s_x + 4 * (i + (i >> 2))) = xv[v];
    }
    __syncthreads();
#pragma unroll
    for (int s = 0; s < CPL; ++s) {
      const int c = cval[s] ? s * 64 * wk + kw * 64 + lane : 0;
#pragma unroll
      for (int m = 0; m < M; ++m)
#pragma unroll
        for (int qi = 0; qi < CX / 4; ++qi) {
          const int vi = ((m * k_cols + c * CW) >> 3) + qi;    // 16-byte vector index
          u32x4 v = *reinterpret_cast<const u32x4*>(s_x + 4 * (vi + (vi >> 2)));
          if (!cval[s]) v = 0;
          xr[m][s][4 * qi] = v.x; xr[m][s][4 * qi + 1] = v.y;
          xr[m][s][4 * qi + 2] = v.z; xr[m][s][4 * qi + 3] = v.w;
        }
    }
  } else if (SPLITK) {
    direct_x();
  }

  float acc[M];
  __syncthreads();  // pair table and ticket counter ready (and, when staged, x read out of LDS)
  if constexpr (!SPLITK && !kRestAfterFill) {
#pragma unroll
    for (int b = 1; b < NBUF; ++b) load_row(rq[b], q[b]);
  }

  if constexpr (!SPLITK) {
    float res[M];        // lane i: results of the wavefront's i-th held row
    int res_row = n_rows;
    int held = 0;
#pragma unroll
    for (int m = 0; m < M; ++m) res[m] = 0.0f;
    auto flush = [&]() {
      if (lane < held && res_row < n_rows) {
#pragma unroll
        for (int m = 0; m < M; ++m) y[(int64_t)m * n_rows + res_row] = res[m];
      }
      held = 0;
    };
    // One slot: ask for the next ticket (when rows remain), compute the row in buffer b, then
    // load the ticket's row into b. The ticket is read only after the row's products (the asm
    // ties it to their sum): an earlier read would make the wavefront wait for the LDS lookups.
    auto step = [&](int b) {
      const int newest = rq[(b + NBUF - 1) % NBUF];
      uint32_t tk = 0;
      if (newest < n_rows && lane == 0)
        tk = __hip_atomic_fetch_add(&s_ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      float dep = 0.0f;
      if (rq[b] < n_rows) {
        gemv_row<BITS, M, CPL>(q[b], xr, s_lut, laneoff, acc);
#pragma unroll
        for (int m = 0; m < M; ++m) {
          const float t = wave_sum(acc[m]) * scale;
          res[m] = (lane == held) ? t : res[m];
          dep += t;
        }
        res_row = (lane == held) ? rq[b] : res_row;
        if (++held == 64) flush();
      }
      uint32_t tks;
      asm volatile("v_readfirstlane_b32 %0, %1" : "=s"(tks) : "v"(tk), "v"(dep));
      rq[b] = newest < n_rows ? ticket_row(tks) : n_rows;
      load_row(rq[b], q[b]);
    };
    // Rows come in increasing order, so once the oldest buffer holds no row, none does.
    while (rq[0] < n_rows) {
#pragma unroll
      for (int b = 0; b < NBUF; ++b) step(b);
    }
    flush();
  } else {
    // Each wavefront leaves its row partials in slot it % kRed of set (it / kRed) % 2; after
    // every kRed rows (and after the last) one barrier, then wavefront kw = 0 of each group sums
    // the WK partials of those rows and stores them. The next kRed rows fill the other set, so
    // no second barrier is needed before a set is written again (its readers have passed the
    // barrier that ends the rows in between).
    auto finish_row = [&](int it) {
      const int slot = it % kRed, set = (it / kRed) & 1;
#pragma unroll
      for (int m = 0; m < M; ++m) {
        const float t = wave_sum(acc[m]);
        if (lane == 0) s_part[set][slot][wave][m] = t;
      }
      if (slot == kRed - 1 || it == iters - 1) {
        __syncthreads();
        if (kw == 0 && lane < kRed * M) {
          const int sl = lane / M, m = lane % M;
          const int it2 = it - slot + sl;
          const int r = gid + it2 * total_groups;
          if (sl <= slot && r < n_rows) {
            float t = 0.0f;
            for (int w2 = 0; w2 < wk; ++w2) t += s_part[set][sl][grp * wk + w2][m];
            y[(int64_t)m * n_rows + r] = t * scale;
          }
        }
      }
    };
#pragma unroll
    for (int b = 1; b + 1 < NBUF; ++b) load_row(gid + b * total_groups, q[b]);
    // Invariant at the top of the loop: q[b] holds (or awaits) row it + b for b < NBUF - 1.
    int it = 0;
    for (; it + NBUF <= iters; it += NBUF) {
#pragma unroll
      for (int b = 0; b < NBUF; ++b) {
        load_row(gid + (it + b + NBUF - 1) * total_groups, q[(b + NBUF - 1) % NBUF]);
        gemv_row<BITS, M, CPL>(q[b], xr, s_lut, laneoff, acc);
        finish_row(it + b);
      }
    }
#pragma unroll
    for (int b = 0; b + 1 < NBUF; ++b) {
      if (it + b < iters) {
        gemv_row<BITS, M, CPL>(q[b], xr, s_lut, laneoff, acc);
        finish_row(it + b);
      }
    }
  }
}

// ------------------------------------------------------------------ GPTQ calibration
//
// Rows of W evolve independently given U, so the column loop runs one wavefront per row: lane
// l holds columns i1 + l and i1 + 64 + l of the current block. Column i's value is read across
// the wavefront (v_readlane), quantized to the fixed codebook by threshold counting (the same
// decision as the encoders), and err = (w - q) / U_ii is subtracted, times U_ij, from the
// block's later columns held by the lanes; the block's rows of U sit in LDS. After the block a
// second kernel subtracts sum_i err_i U_ij from every later column (16 rows x 64 columns per
// workgroup, the block's errors and U rows staged in LDS). Every operation is a separately
// rounded float32 operation in a fixed order (no contraction), which fixes the result bits.
constexpr int kGptqBlock = 128;

struct GptqQuant {
  float cb[16];      // value of each code
  float th[15];      // LogbQuant: 7 magnitude thresholds on |w|; baseline: 15 on w
  int uniform;       // 0: sign + magnitude (LogbQuant), 1: unsigned code (baseline)
};

__device__ __forceinline__ uint32_t gptq_code(float w, const GptqQuant& qz) {
  uint32_t c = 0;
  if (qz.uniform) {
#pragma unroll
    for (int t = 0; t < 15; ++t) c += (w >= qz.th[t]) ? 1u : 0u;
  } else {
    const float a = __builtin_fabsf(w);
#pragma unroll
    for (int t = 0; t < 7; ++t) c += (a >= qz.th[t]) ? 1u : 0u;
    if (w < 0.0f && c != 0u) c |= 8u;
  }
  return c;
}

__global__ __launch_bounds__(512) void k_gptq_panel(float* __restrict__ w, int n_rows, int k_cols,
                                                    const float* __restrict__ u, int i1, int nb,
                                                    GptqQuant qz, float* __restrict__ err,
                                                    uint8_t* __restrict__ codes) {
#pragma clang fp contract(off)
  __shared__ float s_u[kGptqBlock * kGptqBlock];
  for (int idx = threadIdx.x; idx < nb * nb; idx += 512) {
    const int a = idx / nb, b = idx % nb;
    s_u[a * kGptqBlock + b] = u[(int64_t)(i1 + a) * k_cols + i1 + b];
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 8 + (threadIdx.x >> 6);
  if (row >= n_rows) return;
  float* wr = w + (int64_t)row * k_cols + i1;
  float p0 = lane < nb ? wr[lane] : 0.0f;
  float p1 = 64 + lane < nb ? wr[64 + lane] : 0.0f;
  uint32_t c0 = 0, c1 = 0;
  for (int i = 0; i < nb; ++i) {
    const float wi = __builtin_bit_cast(float, __builtin_amdgcn_readlane(
        __builtin_bit_cast(int, i < 64 ? p0 : p1), i & 63));
    const uint32_t c = gptq_code(wi, qz);
    const float e = __fdiv_rn(wi - qz.cb[c], s_u[i * kGptqBlock + i]);
    if (lane == (i & 63)) {
      if (i < 64) c0 = c; else c1 = c;
    }
    if (lane == 0) err[(int64_t)row * kGptqBlock + i] = e;
    const float* ui = s_u + i * kGptqBlock;
    if (lane > i && lane < nb) p0 = p0 - e * ui[lane];
    if (64 + lane > i && 64 + lane < nb) p1 = p1 - e * ui[64 + lane];
  }
  if (lane < nb) wr[lane] = p0;
  if (64 + lane < nb) wr[64 + lane] = p1;
  // Byte b of the block holds columns 2b (low nibble) and 2b + 1.
  const int src = (2 * lane) & 63;
  const uint32_t lo0 = __builtin_amdgcn_ds_bpermute(src << 2, (int)c0);
  const uint32_t hi0 = __builtin_amdgcn_ds_bpermute((src + 1) << 2, (int)c0);
  const uint32_t lo1 = __builtin_amdgcn_ds_bpermute(src << 2, (int)c1);
  const uint32_t hi1 = __builtin_amdgcn_ds_bpermute((src + 1) << 2, (int)c1);
  const uint32_t byte = lane < 32 ? (lo0 | (hi0 << 4)) : (lo1 | (hi1 << 4));
  if (2 * lane < nb) codes[(int64_t)row * (k_cols / 2) + i1 / 2 + lane] = (uint8_t)byte;
}

__global__ __launch_bounds__(256) void k_gptq_trail(float* __restrict__ w, int n_rows, int k_cols,
                                                    const float* __restrict__ u, int i1, int nb,
                                                    const float* __restrict__ err) {
#pragma clang fp contract(off)
  __shared__ float s_e[16][kGptqBlock];
  __shared__ __attribute__((aligned(16))) float s_u[kGptqBlock][64];
  const int i2 = i1 + nb;
  const int r0 = blockIdx.y * 16;
  const int c0 = i2 + blockIdx.x * 64;
  for (int idx = threadIdx.x; idx < 16 * kGptqBlock; idx += 256) {
    const int r = idx / kGptqBlock, i = idx % kGptqBlock;
    s_e[r][i] = (r0 + r < n_rows && i < nb) ? err[(int64_t)(r0 + r) * kGptqBlock + i] : 0.0f;
  }
  for (int idx = threadIdx.x; idx < kGptqBlock * 64; idx += 256) {
    const int i = idx / 64, c = idx % 64;
    s_u[i][c] = (i < nb && c0 + c < k_cols) ? u[(int64_t)(i1 + i) * k_cols + c0 + c] : 0.0f;
  }
  __syncthreads();
  const int r = threadIdx.x >> 4;          // 16 rows
  const int cq = (threadIdx.x & 15) * 4;   // 4 columns each
  float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int i = 0; i < nb; ++i) {
    const float e = s_e[r][i];
    const f32x4 uv = *reinterpret_cast<const f32x4*>(&s_u[i][cq]);
    acc[0] = acc[0] + e * uv.x;
    acc[1] = acc[1] + e * uv.y;
    acc[2] = acc[2] + e * uv.z;
    acc[3] = acc[3] + e * uv.w;
  }
  const int row = r0 + r;
  if (row >= n_rows) return;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int col = c0 + cq + q;
    if (col < k_cols) {
      float* p = w + (int64_t)row * k_cols + col;
      *p = *p - acc[q];
    }
  }
}

// ------------------------------------------------------------------ MFMA skinny GEMM, register dequant
//
// For sign-symmetric codebooks (codebook[8 + k] = -codebook[k], codebook[k] >= 0 for k < 8,
// which every fitted codebook is) a code dword is dequantized in registers: the magnitude
// nibbles index 8-byte tables of the float16 low and high bytes with v_perm_b32, the sign bits
// are OR-ed into the high bytes, and four more v_perm_b32 assemble the float16 pairs. The B
// operand then holds the eight weights of the dword in the order k0 k2 k4 k6 k1 k3 k5 k7; the
// activation tile is written to LDS in that same order, so each MFMA still contracts matching
// (x, w) pairs. Without the 64 KiB pair table, LDS holds a ring of activation tiles and the
// codes of STAGES steps stay in flight per wavefront.
//
// Tiling: v_mfma_f32_16x16x32_f16 with the activations as A (16 batch rows x 32 K) and the
// weights as B (32 K x 16 weight rows). A workgroup of 8 wavefronts owns 128 weight rows
// (16 per wavefront) and MT * 16 batch rows; every wavefront walks the whole K in steps of
// 256. Lane (j = l % 16, g = l / 16) owns weight row n0 + j and loads code bytes
// [128 step + 32 g, +32), i.e. k in [256 step + 64 g, +64): eight dwords, one per MFMA.
// MFMA d multiplies, for lanes g, k = 256 step + 64 g + 8 d + 0..7; the A operand of lane
// (i, g) is x[i][256 step + 64 g + 8 d .. +8] from the LDS tile (same within-8 order).
// Activation tiles of STAGES - 1 steps ahead sit in an LDS ring; codes of STAGES - 1 steps
// ahead are in flight in registers.
struct LutBytes { uint32_t lo0, lo1, hi0, hi1; };   // float16 bytes of magnitudes 0..3 / 4..7

constexpr int kM2Step = 256;
constexpr int kM2Pad = kM2Step + 8;   // halves per staged activation row

__device__ __forceinline__ void dequant_dword(uint32_t w, const LutBytes& t, uint32_t (&o)[4]) {
  const uint32_t me = w & 0x07070707u;            // magnitudes of k0 k2 k4 k6
  const uint32_t mo = (w >> 4) & 0x07070707u;     // magnitudes of k1 k3 k5 k7
  const uint32_t le = __builtin_amdgcn_perm(t.lo1, t.lo0, me);
  const uint32_t lo = __builtin_amdgcn_perm(t.lo1, t.lo0, mo);
  const uint32_t he = __builtin_amdgcn_perm(t.hi1, t.hi0, me) | ((w << 4) & 0x80808080u);
  const uint32_t ho = __builtin_amdgcn_perm(t.hi1, t.hi0, mo) | (w & 0x80808080u);
  o[0] = __builtin_amdgcn_perm(he, le, 0x05010400u);   // (k0, k2)
  o[1] = __builtin_amdgcn_perm(he, le, 0x07030602u);   // (k4, k6)
  o[2] = __builtin_amdgcn_perm(ho, lo, 0x05010400u);   // (k1, k3)
  o[3] = __builtin_amdgcn_perm(ho, lo, 0x07030602u);   // (k5, k7)
}

// Eight activations x0..x7 (four float16 pairs) reordered to x0 x2 x4 x6 x1 x3 x5 x7.
__device__ __forceinline__ u32x4 permute_x8(const u32x4 v) {
  u32x4 o;
  o.x = __builtin_amdgcn_perm(v.y, v.x, 0x05040100u);
  o.y = __builtin_amdgcn_perm(v.w, v.z, 0x05040100u);
  o.z = __builtin_amdgcn_perm(v.y, v.x, 0x07060302u);
  o.w = __builtin_amdgcn_perm(v.w, v.z, 0x07060302u);
  return o;
}

// LDS position (in 16-byte units) of unit u of staged activation row r: rows 8..15 of every
// 16-row tile are rotated by 8 units, so that the 32 lanes served together by a 128-bit LDS
// read (rows 0..15 x two k-groups 8 units apart) hit 32 distinct bank groups (measured
// conflict-free with SQ_LDS_BANK_CONFLICT; the unrotated padded layout is not).
__device__ __forceinline__ int x_unit(int r, int u) { return (u + 8 * ((r >> 3) & 1)) & 31; }

// PAIRS selects the dequantization: true = the LDS pair table (one v_perm_b32 address and one
// ds_read_b32 per two weights; activations in natural order), false = the register tables
// above (no LDS table, 14 VALU instructions per eight weights; activations permuted).
//
// COAL selects how codes reach the lanes. false: every lane loads its own 32 bytes (two 16-byte
// pieces 32 bytes apart per row and instruction). true: the wavefront reads its 16 rows as two
// instructions of 8 rows x 128 contiguous bytes each, writes them to a private LDS buffer and
// reads them back in the MFMA layout (same wavefront, so no workgroup barrier). On MI355X a
// pure streaming read of 8 rows x 128 B per instruction runs at about 5.9 TB/s, of 16 rows x
// 64 B at about 4.6 TB/s. With COAL the activation tile of a step is also requested together
// with that step's codes, STAGES - 1 steps ahead: vector loads complete in issue order, so an
// activation load issued later than a code load would wait for it. COAL is used for MT <= 2,
// where it measured 10-20 % faster; larger MT keep the first scheme.
//
// W is the number of wavefronts per workgroup (16 W weight rows). k_mfma2 runs W = 8;
// k_mfma2_narrow runs W = 4 for layers whose 64-row workgroups all fit on the chip at once:
// there every workgroup has a CU to itself either way, and halving the rows per workgroup
// halves the K walk each CU does for the layer.
template <int BITS, int MT, int STAGES, bool PAIRS, bool COAL, int W>
__device__ __forceinline__ void mfma2_body(const uint8_t* __restrict__ codes,
                                           const uint16_t* __restrict__ x,
                                           float* __restrict__ y, int n_rows, int k_cols,
                                           int m_rows, LutBytes tb,
                                           const typename LutOf<BITS>::type& lut, float scale) {
  static_assert(STAGES % 2 == 0, "the loop is unrolled by STAGES and alternates two tiles");
  static_assert(BITS == 4 || PAIRS, "8-bit codes are dequantized through the LDS table");
  static_assert(W == 8 || W == 4, "8 or 4 wavefronts");
  // K parts: workgroup z of gridDim.z takes the steps [z per_z, +per_z) (the last part may be
  // shorter) and adds its partial products into y, which the host has zeroed. The host splits
  // K in at most two parts, so every output receives exactly two adds and 0 + a + b rounds the
  // same in either order.
  const int nsteps_all = (k_cols + kM2Step - 1) / kM2Step;
  const int per_z = (nsteps_all + (int)gridDim.z - 1) / (int)gridDim.z;
  const int s_lo = (int)blockIdx.z * per_z;
  const int nsteps = per_z < nsteps_all - s_lo ? per_z : nsteps_all - s_lo;
  if (nsteps <= 0) return;
  constexpr int NT = 64 * W;             // threads
  constexpr int ROWS = 16 * W;           // weight rows per workgroup
  constexpr int XV = MT * 512 / NT;      // activation vectors per thread per step
  constexpr int RB = 32 * BITS;          // code bytes of one row per step (256 k)
  constexpr int CB = RB / 64;            // 16-byte pieces per lane per step
  constexpr int TP = RB + 16;            // transpose buffer pitch (bytes)
  __shared__ __attribute__((aligned(16))) uint16_t s_x[2][MT * 16][kM2Pad];
  __shared__ __attribute__((aligned(16))) uint32_t s_lut[PAIRS ? kLutWords : 4];
  __shared__ __attribute__((aligned(16))) uint8_t s_ct[COAL ? W * 16 * TP : 16];
  if (PAIRS) fill_lut<BITS, NT>(s_lut, lut);
  const uint32_t laneoff = (uint32_t)(threadIdx.x & 63) << 2;

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = t >> 6;
  const int j = lane & 15;
  const int g = lane >> 4;
  const int n0 = blockIdx.x * ROWS + wave * 16;
  const int mb = blockIdx.y * (MT * 16);
  const int64_t row_bytes = (int64_t)k_cols * BITS / 8;
  // One buffer descriptor over the workgroup's rows (rows past n_rows read as zeros and are
  // not stored). Buffer loads keep the code prefetch where it is issued: plain loads of the
  // read-only codes were moved by the compiler next to their use.
  const int band0 = blockIdx.x * ROWS;
  const int band_rows = n_rows - band0 < ROWS ? n_rows - band0 : ROWS;
  const __amdgpu_buffer_rsrc_t crs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(codes + (int64_t)band0 * row_bytes), (short)0, (int)(band_rows * row_bytes),
      kBufferRsrcWord3);
  const int row = n0 + j;
  const int crow = (wave * 16 + j) * (int)row_bytes;   // this lane's row in the descriptor

  // Steps below are counted within the workgroup's K part (global step s_lo + step).
  // Activation tile of a step: MT*16 rows x 256 halves = MT*512 vectors of 16 bytes, XV per
  // thread. Loads are clamped in bounds; entries past m_rows / k_cols are zeroed when written.
  auto load_x = [&](int step, u32x4 (&v)[XV]) {
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int idx = t + NT * i;
      const int m = mb + (idx >> 5);
      const int kk = (s_lo + step) * kM2Step + (idx & 31) * 8;
      const int mc = m < m_rows ? m : m_rows - 1;
      const int kc = kk < k_cols ? kk : k_cols - 8;
      v[i] = *(GlobalU32x4)((const __attribute__((address_space(1))) uint16_t*)x +
                            (int64_t)mc * k_cols + kc);
    }
  };
  auto store_x = [&](int step, int slot, const u32x4 (&v)[XV]) {
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int idx = t + NT * i;
      const uint32_t keep = 0u - (uint32_t)((mb + (idx >> 5) < m_rows) &
                                            ((s_lo + step) * kM2Step + (idx & 31) * 8 < k_cols));
      u32x4 w = PAIRS ? v[i] : permute_x8(v[i]);
      w.x &= keep; w.y &= keep; w.z &= keep; w.w &= keep;
      const int r = idx >> 5;
      *reinterpret_cast<u32x4*>(&s_x[slot][r][x_unit(r, idx & 31) * 8]) = w;
    }
  };
  // Codes of a step: this lane's RB / 4 bytes at [RB step + (RB / 4) g, +RB / 4) of row n0 + j
  // (clamped into the row; a clamped chunk only meets zero activations), i.e. k in
  // [256 step + 64 g, +64). Without COAL they are loaded as CB 16-byte pieces per lane; with
  // COAL the wavefront loads its rows n0 .. n0 + 15 as CB instructions of RPI rows x RB
  // contiguous bytes (lane l: row n0 + RPI c + l / (RB / 16), bytes 16 (l % (RB / 16))), and
  // lane_codes() redistributes them through the wavefront's LDS buffer.
  constexpr int RPI = 1024 / RB;          // rows per coalesced instruction
  auto load_codes = [&](int step, u32x4 (&q)[CB]) {
#pragma unroll
    for (int c = 0; c < CB; ++c) {
      if (COAL) {
        const int r = wave * 16 + RPI * c + lane / (RB / 16);
        int off = (s_lo + step) * RB + 16 * (lane % (RB / 16));
        off = off + 16 <= (int)row_bytes ? off : (int)row_bytes - 16;
        q[c] = __builtin_amdgcn_raw_buffer_load_b128(crs, r * (int)row_bytes + off, 0,
                                                     kCachePolicyNT);
      } else {
        int off = (s_lo + step) * RB + (RB / 4) * g + 16 * c;
        off = off + 16 <= (int)row_bytes ? off : (int)row_bytes - 16;
        q[c] = __builtin_amdgcn_raw_buffer_load_b128(crs, crow + off, 0, kCachePolicyNT);
      }
    }
  };
  uint8_t* s_cw = s_ct + (COAL ? wave * 16 * TP : 0);
  auto lane_codes = [&](const u32x4 (&q)[CB], u32x4 (&o)[CB]) {
    if (!COAL) {
#pragma unroll
      for (int c = 0; c < CB; ++c) o[c] = q[c];
      return;
    }
    // LDS operations of one wavefront complete in order, so the reads below see the writes.
#pragma unroll
    for (int c = 0; c < CB; ++c)
      *reinterpret_cast<u32x4*>(s_cw + (RPI * c + lane / (RB / 16)) * TP + 16 * (lane % (RB / 16))) = q[c];
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int c = 0; c < CB; ++c)
      o[c] = *reinterpret_cast<const u32x4*>(s_cw + j * TP + (RB / 4) * g + 16 * c);
    __builtin_amdgcn_wave_barrier();
  };

  float4v acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[mt][r] = 0.0f;

  // Pipeline. Activation tile t lives in LDS slot t & 1 and is written there at the end of step
  // t - 1. Codes of step t are loaded at step t - (STAGES - 1) into q[t % STAGES]. Without COAL
  // the tile is loaded at step t - 2 into xr[t & 1]; with COAL at step t - (STAGES - 1) into
  // xr[t % STAGES] (XR = STAGES register sets), so waiting for it never waits for a code load
  // issued after an older tile.
  constexpr int XR = COAL ? STAGES : 2;
  u32x4 q[STAGES][CB];
  u32x4 xr[XR][XV];
  auto clampstep = [&](int t2) { return t2 < nsteps ? t2 : nsteps - 1; };
  if (COAL) {
#pragma unroll
    for (int t2 = 0; t2 < STAGES - 1; ++t2) {
      load_x(clampstep(t2), xr[t2 % XR]);
      load_codes(clampstep(t2), q[t2]);
    }
  } else {
    load_x(0, xr[0]);
    load_x(clampstep(1), xr[1 % XR]);
#pragma unroll
    for (int t2 = 0; t2 < STAGES - 1; ++t2) load_codes(clampstep(t2), q[t2]);
  }
  store_x(0, 0, xr[0]);
  __syncthreads();

  // Steady state, unrolled by STAGES (even) so every buffer index is static.
  for (int s0 = 0; s0 < nsteps; s0 += STAGES) {
#pragma unroll
    for (int u = 0; u < STAGES; ++u) {
      const int step = s0 + u;
      if (step >= nsteps) break;
      if (COAL) load_x(clampstep(step + STAGES - 1), xr[(u + STAGES - 1) % XR]);
      else load_x(clampstep(step + 2), xr[u % XR]);
      load_codes(clampstep(step + STAGES - 1), q[(u + STAGES - 1) % STAGES]);
      u32x4 qc[CB];
      lane_codes(q[u], qc);
      uint32_t dws[4 * CB];
#pragma unroll
      for (int c = 0; c < CB; ++c) {
        dws[4 * c] = qc[c].x; dws[4 * c + 1] = qc[c].y;
        dws[4 * c + 2] = qc[c].z; dws[4 * c + 3] = qc[c].w;
      }
      // MFMA d multiplies k = 256 step + 64 g + 8 d + 0..7: code dword d (4-bit) or dwords
      // 2 d, 2 d + 1 (8-bit).
#pragma unroll
      for (int d = 0; d < 8; ++d) {
        uint32_t bw[4];
        if (BITS == 8) {
          bw[0] = single_pair(s_lut, dws[2 * d], laneoff, 0);
          bw[1] = single_pair(s_lut, dws[2 * d], laneoff, 1);
          bw[2] = single_pair(s_lut, dws[2 * d + 1], laneoff, 0);
          bw[3] = single_pair(s_lut, dws[2 * d + 1], laneoff, 1);
        } else if (PAIRS) {
#pragma unroll
          for (int i = 0; i < 4; ++i) bw[i] = pair_lookup(s_lut, dws[d], laneoff, i);
        } else {
          dequant_dword(dws[d], tb, bw);
        }
        const half8v b = __builtin_bit_cast(half8v, u32x4{bw[0], bw[1], bw[2], bw[3]});
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const half8v a = *reinterpret_cast<const half8v*>(
              &s_x[u & 1][mt * 16 + j][x_unit(j, 8 * g + d) * 8]);
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, acc[mt], 0, 0, 0);
        }
      }
      store_x(step + 1, (u + 1) & 1, xr[(u + 1) % XR]);
      __syncthreads();
    }
  }

#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = mb + mt * 16 + 4 * g + r;
      if (m < m_rows && row < n_rows) {
        if (gridDim.z > 1) unsafeAtomicAdd(&y[(int64_t)m * n_rows + row], acc[mt][r] * scale);
        else y[(int64_t)m * n_rows + row] = acc[mt][r] * scale;
      }
    }
}

template <int BITS, int MT, int STAGES, bool PAIRS, bool COAL>
__global__ __launch_bounds__(512) void k_mfma2(const uint8_t* __restrict__ codes,
                                               const uint16_t* __restrict__ x,
                                               float* __restrict__ y, int n_rows, int k_cols,
                                               int m_rows, LutBytes tb,
                                               typename LutOf<BITS>::type lut, float scale) {
  mfma2_body<BITS, MT, STAGES, PAIRS, COAL, 8>(codes, x, y, n_rows, k_cols, m_rows, tb, lut,
                                               scale);
}

template <int BITS, int MT, bool PAIRS, bool COAL>
__global__ __launch_bounds__(256) void k_mfma2_narrow(const uint8_t* __restrict__ codes,
                                                      const uint16_t* __restrict__ x,
                                                      float* __restrict__ y, int n_rows,
                                                      int k_cols, int m_rows, LutBytes tb,
                                                      typename LutOf<BITS>::type lut,
                                                      float scale) {
  mfma2_body<BITS, MT, 4, PAIRS, COAL, 4>(codes, x, y, n_rows, k_cols, m_rows, tb, lut, scale);
}

// ------------------------------------------------------------------ MFMA GEMM, K quarters, m > 96
//
// For large batches k_mfma2's wavefronts (16 weight rows, every batch tile) re-read a fresh
// activation fragment from LDS for every MFMA. Here a workgroup of 8 wavefronts still owns
// 128 weight rows x 128 batch rows and walks K in steps of 256, but wavefront w takes weight
// rows 64 (w % 2) .. +64 (four 16-row tiles) and the K quarter [256 step + 64 (w / 2), +64) of
// every step, for all eight batch tiles: each activation fragment read from LDS feeds four
// MFMAs and each dequantized weight fragment eight, and no code is loaded or dequantized twice.
// The activation tile is staged through LDS as in k_mfma2 (same rotated layout); within its
// quarter, lane (j, g) holds k in [.. + 16 g, +16) of its rows, i.e. MFMA c contracts
// k = 256 step + 64 kq + 16 g + 8 c + 0..7 (code dword c of the lane's 8 bytes, activation unit
// 8 kq + 2 g + c). The next batch tile's fragment is read while the current tile's four MFMAs
// run. At the end the four K quarters are summed through LDS in a fixed order ((q0 + q2) +
// (q1 + q3)), so results are deterministic. Measured on MI355X (8192 -> 28672): 86.8 us vs
// 96.4 us for k_mfma2 at m = 128, 164 vs 183 us at m = 256; SQ_VALU_MFMA_BUSY_CYCLES puts the
// MFMA pipes at about a third of the kernel's cycles, the rest going to the dequantization and
// staging VALU work, LDS and the per-step barrier.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef const __attribute__((address_space(1))) u32x2* GlobalU32x2;

__global__ __launch_bounds__(512) void k_mfma_kq(const uint8_t* __restrict__ codes,
                                                 const uint16_t* __restrict__ x,
                                                 float* __restrict__ y, int n_rows, int k_cols,
                                                 int m_rows, LutBytes tb, float scale) {
  constexpr int XV = 8;                  // 16-byte activation vectors per thread per step
  __shared__ __attribute__((aligned(16))) uint16_t s_x[2][128][kM2Pad];
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = t >> 6;
  const int j = lane & 15;
  const int g = lane >> 4;
  const int wq = wave & 1;               // weight rows 64 wq .. +64 of the workgroup's 128
  const int kq = wave >> 1;              // k in [256 step + 64 kq, +64) of every step
  const int nb = blockIdx.x * 128 + 64 * wq;
  const int mb = blockIdx.y * 128;
  const int nsteps = (k_cols + kM2Step - 1) / kM2Step;
  const int64_t row_bytes = (int64_t)k_cols / 2;
  // One buffer descriptor over the workgroup's 128 rows (rows past n_rows read as zeros; their
  // results are not stored). Buffer loads keep their place in the program: plain loads of the
  // read-only codes were moved by the compiler next to their use, past the barrier that ends
  // the step before, which took away the one-step prefetch.
  const int band0 = blockIdx.x * 128;
  const int band_rows = n_rows - band0 < 128 ? n_rows - band0 : 128;
  const __amdgpu_buffer_rsrc_t crs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(codes + (int64_t)band0 * row_bytes), (short)0, (int)(band_rows * row_bytes),
      kBufferRsrcWord3);
  int crow[4];
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) crow[rt] = (64 * wq + 16 * rt + j) * (int)row_bytes;
  // Activation tile: as k_mfma2 (clamped loads; rows past m_rows and k past k_cols are zeroed
  // when written to LDS).
  auto load_x = [&](int step, u32x4 (&v)[XV]) {
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int idx = t + 512 * i;
      const int m = mb + (idx >> 5);
      const int kk = step * kM2Step + (idx & 31) * 8;
      const int mc = m < m_rows ? m : m_rows - 1;
      const int kc = kk < k_cols ? kk : k_cols - 8;
      v[i] = *(GlobalU32x4)((const __attribute__((address_space(1))) uint16_t*)x +
                            (int64_t)mc * k_cols + kc);
    }
  };
  auto store_x = [&](int step, int slot, const u32x4 (&v)[XV]) {
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int idx = t + 512 * i;
      const uint32_t keep = 0u - (uint32_t)((mb + (idx >> 5) < m_rows) &
                                            (step * kM2Step + (idx & 31) * 8 < k_cols));
      u32x4 w = permute_x8(v[i]);
      w.x &= keep; w.y &= keep; w.z &= keep; w.w &= keep;
      const int r = idx >> 5;
      *reinterpret_cast<u32x4*>(&s_x[slot][r][x_unit(r, idx & 31) * 8]) = w;
    }
  };
  // Codes of a step for row tile rt: lane (j, g) takes the 8 bytes of k in
  // [256 step + 64 kq + 16 g, +16) of row nb + 16 rt + j (clamped into the row; a clamped piece
  // only meets zero activations).
  auto load_codes = [&](int step, u32x2 (&q)[4]) {
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
      int off = step * 128 + 32 * kq + 8 * g;
      off = off + 8 <= (int)row_bytes ? off : (int)row_bytes - 8;
      q[rt] = __builtin_amdgcn_raw_buffer_load_b64(crs, crow[rt] + off, 0, kCachePolicyNT);
    }
  };
  float4v acc[8][4];
#pragma unroll
  for (int bt = 0; bt < 8; ++bt)
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[bt][rt][r] = 0.0f;

  // Pipeline: activation tile s is loaded into registers during step s - 2 and written to LDS
  // slot s & 1 at the end of step s - 1; the codes of step s are loaded during step s - 1.
  u32x2 q[2][4];
  u32x4 xr[XV];
  auto clampstep = [&](int t2) { return t2 < nsteps ? t2 : nsteps - 1; };
  load_x(0, xr);
  load_codes(0, q[0]);
  store_x(0, 0, xr);
  load_x(clampstep(1), xr);
  __syncthreads();

  for (int s0 = 0; s0 < nsteps; s0 += 2) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int step = s0 + u;
      if (step >= nsteps) break;
      load_codes(clampstep(step + 1), q[u ^ 1]);
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        half8v b[4];
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
          uint32_t bw[4];
          dequant_dword(c == 0 ? q[u][rt].x : q[u][rt].y, tb, bw);
          b[rt] = __builtin_bit_cast(half8v, u32x4{bw[0], bw[1], bw[2], bw[3]});
        }
        const uint16_t* abase = &s_x[u][j][x_unit(j, 8 * kq + 2 * g + c) * 8];
        half8v a_cur = *reinterpret_cast<const half8v*>(abase);
#pragma unroll
        for (int bt = 0; bt < 8; ++bt) {
          half8v a_nxt = a_cur;
          if (bt + 1 < 8) a_nxt = *reinterpret_cast<const half8v*>(abase + 16 * (bt + 1) * kM2Pad);
#pragma unroll
          for (int rt = 0; rt < 4; ++rt)
            acc[bt][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a_cur, b[rt], acc[bt][rt], 0, 0, 0);
          a_cur = a_nxt;
        }
      }
      store_x(step + 1, u ^ 1, xr);
      load_x(clampstep(step + 2), xr);
      __syncthreads();
    }
  }

  // Sum the four K quarters through LDS (the activation slots are free after the last
  // barrier): quarters 2, 3 are added to 0, 1, then 1 to 0, which stores. Each of the four
  // slots holds one wavefront's 8 x 4 tiles (8192 floats).
  float* s_red = reinterpret_cast<float*>(&s_x[0][0][0]);
  static_assert(sizeof(s_x) >= 4 * 8192 * sizeof(float), "reduction slots fit the tile buffers");
  auto red_slot = [&](int w_q, int half) { return s_red + (size_t)(w_q * 2 + half) * 8192; };
  auto put = [&](float* dst) {
#pragma unroll
    for (int bt = 0; bt < 8; ++bt)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt)
        *reinterpret_cast<float4v*>(dst + ((bt * 4 + rt) * 64 + lane) * 4) = acc[bt][rt];
  };
  __syncthreads();
  auto add = [&](const float* src) {
#pragma unroll
    for (int bt = 0; bt < 8; ++bt)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt)
        acc[bt][rt] += *reinterpret_cast<const float4v*>(src + ((bt * 4 + rt) * 64 + lane) * 4);
  };
  if (kq >= 2) put(red_slot(wq, kq - 2));
  __syncthreads();
  if (kq < 2) add(red_slot(wq, kq));
  __syncthreads();
  if (kq == 1) put(red_slot(wq, 0));
  __syncthreads();
  if (kq == 0) {
    add(red_slot(wq, 0));
#pragma unroll
    for (int bt = 0; bt < 8; ++bt)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        const int row = nb + 16 * rt + j;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = mb + 16 * bt + 4 * g + r;
          if (m < m_rows && row < n_rows) y[(int64_t)m * n_rows + row] = acc[bt][rt][r] * scale;
        }
      }
  }
}

// ------------------------------------------------------------------ MFMA GEMM, K quarters, 8-bit
//
// k_mfma_kq on 8-bit codes: a workgroup of 8 wavefronts owns 128 weight rows x 128 batch rows;
// wavefront w takes weight rows 64 (w % 2) .. +64 and the K quarter w / 2 of every step of 128 k,
// for all eight batch tiles, so each weight is looked up once in the LDS table of float16 images
// and feeds 8 MFMAs. Steps of 128 k (not 256) keep two activation slots (2 x 34 KiB) beside the
// 64 KiB table. Lane (j, g) holds k = 128 step + 32 kq + 8 g + 0..7 of its rows (natural order,
// 8 code bytes per row tile). After the last step the table and the slots are reused to sum the
// four K quarters in a fixed order ((q0 + q2) + (q1 + q3)). Measured on MI355X against the
// stepped kernel (8-bit, LDS table): 8192 -> 28672 at m = 128 / 256: 213.9 / 419.1 ->
// 133.4 / 251.3 us; it has only N / 128 workgroups, so narrower layers stay stepped
// (4096 -> 14336 at m = 128: 51.5 vs 70.5 us), and below m = 65 one stepped column wins
// (m = 64: 112.9 vs 129.6 us).
constexpr int kKq8Step = 128;
constexpr int kKq8Pad = kKq8Step + 8;   // halves per staged activation row
__global__ __launch_bounds__(512) void k_mfma_kq8(const uint8_t* __restrict__ codes,
                                                  const uint16_t* __restrict__ x,
                                                  float* __restrict__ y, int n_rows, int k_cols,
                                                  int m_rows, float scale, Lut256 lut) {
  constexpr int XV = 4;                  // 16-byte activation vectors per thread per step
  constexpr int kTableBytes = kLutWords * 4;
  constexpr int kSlotBytes = 128 * kKq8Pad * 2;
  __shared__ __attribute__((aligned(16))) uint8_t s_mem[kTableBytes + 2 * kSlotBytes];
  uint32_t* s_lut = reinterpret_cast<uint32_t*>(s_mem);
  auto slot = [&](int u) { return reinterpret_cast<uint16_t*>(s_mem + kTableBytes + u * kSlotBytes); };
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = t >> 6;
  const int j = lane & 15;
  const int g = lane >> 4;
  const int wq = wave & 1;
  const int kq = wave >> 1;
  const uint32_t laneoff = (uint32_t)lane << 2;
  const int nb = blockIdx.x * 128 + 64 * wq;
  const int mb = blockIdx.y * 128;
  const int nsteps = (k_cols + kKq8Step - 1) / kKq8Step;
  // One buffer descriptor over the workgroup's 128 rows, as in k_mfma_kq (buffer loads keep
  // the one-step code prefetch in place; rows past n_rows read as zeros and are not stored).
  const int band0 = blockIdx.x * 128;
  const int band_rows = n_rows - band0 < 128 ? n_rows - band0 : 128;
  const __amdgpu_buffer_rsrc_t crs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(codes + (int64_t)band0 * k_cols), (short)0, band_rows * k_cols, kBufferRsrcWord3);
  int crow[4];
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) crow[rt] = (64 * wq + 16 * rt + j) * k_cols;
  auto load_x = [&](int step, u32x4 (&v)[XV]) {
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int idx = t + 512 * i;
      const int m = mb + (idx >> 4);
      const int kk = step * kKq8Step + (idx & 15) * 8;
      const int mc = m < m_rows ? m : m_rows - 1;
      const int kc = kk < k_cols ? kk : k_cols - 8;
      v[i] = *(GlobalU32x4)((const __attribute__((address_space(1))) uint16_t*)x +
                            (int64_t)mc * k_cols + kc);
    }
  };
  auto store_x = [&](int step, int u, const u32x4 (&v)[XV]) {
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int idx = t + 512 * i;
      const uint32_t keep = 0u - (uint32_t)((mb + (idx >> 4) < m_rows) &
                                            (step * kKq8Step + (idx & 15) * 8 < k_cols));
      u32x4 w = v[i];
      w.x &= keep; w.y &= keep; w.z &= keep; w.w &= keep;
      *reinterpret_cast<u32x4*>(slot(u) + (idx >> 4) * kKq8Pad + (idx & 15) * 8) = w;
    }
  };
  // Codes of a step for row tile rt: 8 bytes of row nb + 16 rt + j at k = 128 step + 32 kq + 8 g
  // (clamped into the row; a clamped piece only meets zero activations).
  auto load_codes = [&](int step, u32x2 (&q)[4]) {
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
      int off = step * kKq8Step + 32 * kq + 8 * g;
      off = off + 8 <= k_cols ? off : k_cols - 8;
      q[rt] = __builtin_amdgcn_raw_buffer_load_b64(crs, crow[rt] + off, 0, kCachePolicyNT);
    }
  };
  float4v acc[8][4];
#pragma unroll
  for (int bt = 0; bt < 8; ++bt)
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[bt][rt][r] = 0.0f;

  u32x2 q[2][4];
  u32x4 xr[XV];
  auto clampstep = [&](int t2) { return t2 < nsteps ? t2 : nsteps - 1; };
  load_x(0, xr);
  load_codes(0, q[0]);
  fill_single_lut<512>(s_lut, lut);
  store_x(0, 0, xr);
  load_x(clampstep(1), xr);
  __syncthreads();

  for (int s0 = 0; s0 < nsteps; s0 += 2) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int step = s0 + u;
      if (step >= nsteps) break;
      load_codes(clampstep(step + 1), q[u ^ 1]);
      half8v b[4];
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        const u32x4 bw{single_pair(s_lut, q[u][rt].x, laneoff, 0),
                       single_pair(s_lut, q[u][rt].x, laneoff, 1),
                       single_pair(s_lut, q[u][rt].y, laneoff, 0),
                       single_pair(s_lut, q[u][rt].y, laneoff, 1)};
        b[rt] = __builtin_bit_cast(half8v, bw);
      }
      const uint16_t* abase = slot(u) + j * kKq8Pad + 32 * kq + 8 * g;
      half8v a_cur = *reinterpret_cast<const half8v*>(abase);
#pragma unroll
      for (int bt = 0; bt < 8; ++bt) {
        half8v a_nxt = a_cur;
        if (bt + 1 < 8) a_nxt = *reinterpret_cast<const half8v*>(abase + 16 * (bt + 1) * kKq8Pad);
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
          acc[bt][rt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a_cur, b[rt], acc[bt][rt], 0, 0, 0);
        a_cur = a_nxt;
      }
      store_x(step + 1, u ^ 1, xr);
      load_x(clampstep(step + 2), xr);
      __syncthreads();
    }
  }

  // Sum the four K quarters through LDS (table and slots are free after the last barrier).
  float* s_red = reinterpret_cast<float*>(s_mem);
  static_assert(sizeof(s_mem) >= 4 * 8192 * sizeof(float), "reduction slots fit");
  auto red_slot = [&](int w_q, int half) { return s_red + (size_t)(w_q * 2 + half) * 8192; };
  auto put = [&](float* dst) {
#pragma unroll
    for (int bt = 0; bt < 8; ++bt)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt)
        *reinterpret_cast<float4v*>(dst + ((bt * 4 + rt) * 64 + lane) * 4) = acc[bt][rt];
  };
  auto add = [&](const float* src) {
#pragma unroll
    for (int bt = 0; bt < 8; ++bt)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt)
        acc[bt][rt] += *reinterpret_cast<const float4v*>(src + ((bt * 4 + rt) * 64 + lane) * 4);
  };
  if (kq >= 2) put(red_slot(wq, kq - 2));
  __syncthreads();
  if (kq < 2) add(red_slot(wq, kq));
  __syncthreads();
  if (kq == 1) put(red_slot(wq, 0));
  __syncthreads();
  if (kq == 0) {
    add(red_slot(wq, 0));
#pragma unroll
    for (int bt = 0; bt < 8; ++bt)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        const int row = nb + 16 * rt + j;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = mb + 16 * bt + 4 * g + r;
          if (m < m_rows && row < n_rows) y[(int64_t)m * n_rows + row] = acc[bt][rt][r] * scale;
        }
      }
  }
}

// ------------------------------------------------------------------ split-K MFMA, m <= 16
//
// For T batch tiles of 16 rows (T = 1 for m <= 16, T = 2 for m <= 32) and K = 32 W ND KS (W
// wavefronts of ND code dwords per row each, KS workgroups per block): a workgroup of W
// wavefronts takes one block of 16 weight rows at a time (blocks dealt round-robin over the
// grid) and its wavefront w takes the K slice [w S, (w + 1) S), S = 32 ND, of its K part.
// The workgroup therefore streams its 16 rows as one contiguous band, instead of every
// workgroup walking K in step over all rows (measured on MI355X: this code stream reads the
// 8192 x 28672 codes in 20.2 us, the stepped pattern of k_mfma2 in 25 us).
//
// A lane's activations for its slice stay in registers for the whole kernel. With G batch
// groups (G = 1 for m <= 16, G = 2 for m <= 8) the 16 rows of the MFMA's A operand hold G
// copies of the batch rows 0 .. 16 / G - 1, each for a different code dword: lane (j, g)
// holds batch row j % (16 / G) for the dwords d = G r + j / (16 / G), r = 0 .. ND / G - 1,
// at k = w S + 8 ND g + 8 d + 0..7 (zeros for batch rows >= m). MFMA d then leaves correct
// products in the D rows of dword group d % G only and accumulates into that group's tile; the
// other rows are never read. Each lane keeps ND / G activation registers instead of ND, which
// is what lets 16 wavefronts (4 per SIMD) hold K = 8192 at m <= 8.
//
// The codes of a block are loaded as ND / 4 instructions of 64 / ND rows x 16 ND contiguous
// bytes and transposed through the wavefront's LDS buffer so that lane (j, g) then holds row j,
// bytes [4 ND g, 4 ND (g + 1)) of the slice: dword d (k = w S + 8 ND g + 8 d + 0..7) is the B
// operand of MFMA d, matching the A operand above. The 16 x 16 tiles of the W wavefronts and G
// groups are summed in LDS in a fixed order (two sets, one barrier per block); each of the
// first 16 x 16 / G threads owns one (batch row, weight row) element and keeps its results for
// up to 4 blocks before storing them. The next block's codes are in flight while a block is
// computed.
//
// Configurations (measured on MI355X against the 8-wavefront, G = 1 kernel that preceded
// them, same box): K = 8192 takes W = 16, ND = 16 (8192 -> 28672 at m = 4 / 8 / 12:
// 28.1 / 29.5 / 31.3 -> 27.1 / 27.8 / 29.1 us, on another box 27.9 / 29.2 -> 24.6 / 26.3 us);
// K = 4096 takes W = 16, ND = 8 (4096 -> 14336 at m = 4 / 8: 10.1 / 10.5 -> 9.3 / 9.9 us);
// K = 1024 and 2048 keep W = 8. A non-symmetric codebook (the LDS pair table, 64 KiB) keeps
// W = 8 and G = 1. Two batch tiles (17 <= m <= 32, register tables only) hold 2 ND activation
// registers per lane: W = 16 with ND = 4 and 8 at K = 2048 and 4096, W = 8 at K = 1024, and at
// K = 8192 two K parts (KS = 2) of ND = 8: workgroups 2 i and 2 i + 1 take the two K halves of
// the same blocks and add their results into y with float atomics after y is zeroed (two terms
// onto zero: the same sum in either order, so results stay deterministic). The alternative
// of two launches (the second adding into y) measured 7-8 us slower at 8192 -> 28672.
// K = 14336 (m <= 16; G = 2 up to m = 8) takes the same K split over
// workgroup pairs of W = 14 wavefronts, ND = 16: 14336 -> 4096 at m = 4 / 8: 14.5 / 26.7 ->
// 11.5 / 12.6 us against the split-row GEMV and the stepped kernel (one 16-wavefront workgroup
// per block, ND = 28, measured 14.8 / 17.2 us: 256 blocks leave each workgroup one block, with
// nothing to overlap); at m = 9 / 12 / 16: 34.6 / 34.6 / 34.7 -> 13.7-13.9 / 14.7 / 15.8 us
// against the stepped kernel with 64-row workgroups.
//
// Up to kMaxSegs linears that share x, in one launch: their 16-row blocks are numbered one
// after another (segment s holds blocks [blk_begin, blk_begin + ceil(n_rows / 16))), and every
// block is computed exactly as in a launch of its linear alone. Grouped launches need
// sign-symmetric codebooks (register dequantization: each block's tables are its segment's
// kernel arguments); the pair table (PAIRS) serves one segment only.
struct SkSeg {
  const uint8_t* codes;
  float* y;
  int n_rows;
  int blk_begin;
  LutBytes tb;
  float scale;
};
struct SkSegs {
  SkSeg s[kMaxSegs];
};

template <int ND, int WAVES, int G, int T, int KS, bool PAIRS>
__global__ __launch_bounds__(64 * WAVES) void k_mfma_sk(const uint16_t* __restrict__ x,
                                                 const uint8_t* codes0, int n_rows0, int nseg,
                                                 int nblocks, int k_cols, int m_rows,
                                                 SkSegs segs, Lut16 lut) {
  static_assert(ND == 4 || ND == 8 || ND == 16 || ND == 32, "64 / ND rows per load");
  static_assert(G == 1 || G == 2 || G == 4, "batch groups");
  static_assert((T == 1 || (T == 2 && G == 1 && !PAIRS)) && (KS == 1 || (KS == 2 && !PAIRS)),
                "two batch tiles and the K split only with register tables");
  constexpr int BR = 16 * ND;            // code bytes per row per wavefront and block
  constexpr int RPI = 64 / ND;           // rows per load instruction
  constexpr int NI = ND / 4;             // load instructions per block
  constexpr int TP = BR + 16;            // transpose pitch (bytes)
  constexpr int NRES = 4;                // blocks whose results a thread holds before storing
  constexpr int MB = 16 / G;             // batch rows per group
  constexpr int XR = ND / G;             // activation registers per lane and tile
  constexpr int NT = 64 * WAVES;
  constexpr int NOUT = 16 * MB * T;      // outputs per block: batch rows x 16 weight rows
  __shared__ __attribute__((aligned(16))) uint32_t s_lut[PAIRS ? kLutWords : 4];
  __shared__ __attribute__((aligned(16))) uint8_t s_ct[WAVES][16 * TP];
  __shared__ __attribute__((aligned(16))) float4v s_red[2][WAVES][T][64];
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int j = lane & 15, g = lane >> 4;
  const uint32_t laneoff = (uint32_t)lane << 2;
  const int64_t row_bytes = (int64_t)k_cols / 2;
  // K part of this workgroup (KS = 2: workgroups 2 i and 2 i + 1 take the two halves of the
  // same blocks) and its first block.
  const int part = KS == 2 ? (int)(blockIdx.x & 1) : 0;
  const int gb = (int)gridDim.x / KS;
  const int b0 = (int)blockIdx.x / KS;
  const int slice_k0 = part * (k_cols / KS) + w * 32 * ND;
  const int slice_b0 = part * (int)(row_bytes / KS) + w * BR;
  // The fields of the segment that holds block b, selected with static indices: a field read
  // at a run-time segment index compiles to a vector load from the argument block, and its
  // wait would also wait for every code load in flight.
  struct SegView {
    const uint8_t* codes;
    float* y;
    int n_rows, blk_begin;
    LutBytes tb;
    float scale;
  };
  auto seg_view = [&](int b) {
    SegView v{segs.s[0].codes, segs.s[0].y, segs.s[0].n_rows, segs.s[0].blk_begin,
              segs.s[0].tb, segs.s[0].scale};
#pragma unroll
    for (int i = 1; i < kMaxSegs; ++i)
      if (i < nseg && b >= segs.s[i].blk_begin)
        v = SegView{segs.s[i].codes, segs.s[i].y, segs.s[i].n_rows, segs.s[i].blk_begin,
                    segs.s[i].tb, segs.s[i].scale};
    return v;
  };
  // Activations first (they return first): in tile tt, lane row j is batch row
  // 16 tt + j % MB of dword group j / MB; register r holds dword d = G r + j / MB of this
  // lane's slice, in the order the dequantization produces the weights.
  u32x4 xa[T][XR];
#pragma unroll
  for (int tt = 0; tt < T; ++tt) {
    const int mrow = 16 * tt + j % MB, sg = j / MB;
    const bool live = mrow < m_rows;
    const int64_t base = (int64_t)(live ? mrow : 0) * k_cols + slice_k0 + 8 * ND * g;
#pragma unroll
    for (int r = 0; r < XR; ++r)
      xa[tt][r] = *reinterpret_cast<const u32x4*>(x + base + 8 * (G * r + sg));
#pragma unroll
    for (int r = 0; r < XR; ++r) {
      u32x4 v = live ? xa[tt][r] : u32x4{0u, 0u, 0u, 0u};
      xa[tt][r] = PAIRS ? v : permute_x8(v);
    }
  }
  // Codes of block b: a descriptor over its rows (size 0 past the last block, short for a
  // partial last block), so rows past n_rows read as zeros.
  auto load_block = [&](int b, u32x4 (&q)[NI]) {
    const int bb = b < nblocks ? b : nblocks - 1;
    const uint8_t* codes = codes0;
    int n_rows = n_rows0, lb = bb;
    if (nseg > 1) {
      const SegView v = seg_view(bb);
      codes = v.codes;
      n_rows = v.n_rows;
      lb = bb - v.blk_begin;
    }
    const int64_t base = (int64_t)lb * 16 * row_bytes;
    const int64_t avail = (int64_t)n_rows * row_bytes - base;
    const int size = b < nblocks ? (int)(avail < 16 * row_bytes ? avail : 16 * row_bytes) : 0;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(codes + base), (short)0, size, kBufferRsrcWord3);
#pragma unroll
    for (int c = 0; c < NI; ++c) {
      const int r = RPI * c + lane / ND;
      const int off = r * (int)row_bytes + slice_b0 + 16 * (lane % ND);
      q[c] = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, kCachePolicyNT);
    }
  };
  u32x4 q[2][NI];
  load_block(b0, q[0]);
  if constexpr (PAIRS) fill_lut<4, NT>(s_lut, lut);
  __syncthreads();

  float res[NRES];
  int held = 0, blast = 0, par = 0;
  const int ri = t >> 4, rj = t & 15;      // element of threads t < NOUT: batch ri, row rj
  // KS = 2: each output receives exactly two float atomic adds onto zero (the caller zeroes
  // y first), and a + b = b + a, so the result does not depend on their order.
  auto flush = [&]() {
    if (t < NOUT && ri < m_rows) {
#pragma unroll
      for (int h = 0; h < NRES; ++h) {
        if (h < held) {
          const int b = blast - (held - 1 - h) * gb;
          const SegView v = seg_view(b);
          const int n_rows = v.n_rows;
          const int row = (b - v.blk_begin) * 16 + rj;
          if (row < n_rows) {
            float* yp = v.y + (int64_t)ri * n_rows + row;
            if (KS == 2) unsafeAtomicAdd(yp, res[h]);
            else *yp = res[h];
          }
        }
      }
    }
    held = 0;
  };
  uint8_t* s_cw = s_ct[w];
  const int my_group = (lane >> 4) * G / 4;   // dword group of this lane's D rows
  auto block = [&](int b, const u32x4 (&qc)[NI]) {
    const SegView sv = seg_view(b);
    const LutBytes tb = sv.tb;
    const float scale = sv.scale;
    // LDS operations of one wavefront complete in order: the reads see the writes.
#pragma unroll
    for (int c = 0; c < NI; ++c)
      *reinterpret_cast<u32x4*>(s_cw + (RPI * c + lane / ND) * TP + 16 * (lane % ND)) = qc[c];
    __builtin_amdgcn_wave_barrier();
    u32x4 o[NI];
#pragma unroll
    for (int c = 0; c < NI; ++c)
      o[c] = *reinterpret_cast<const u32x4*>(s_cw + j * TP + 4 * ND * g + 16 * c);
    __builtin_amdgcn_wave_barrier();
    float4v acc[T][G];
#pragma unroll
    for (int tt = 0; tt < T; ++tt)
#pragma unroll
      for (int s = 0; s < G; ++s) acc[tt][s] = float4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int d = 0; d < ND; ++d) {
      const u32x4 od = o[d >> 2];
      const uint32_t dw = (d & 3) == 0 ? od.x : (d & 3) == 1 ? od.y : (d & 3) == 2 ? od.z : od.w;
      uint32_t bw[4];
      if (PAIRS) {
#pragma unroll
        for (int i = 0; i < 4; ++i) bw[i] = pair_lookup(s_lut, dw, laneoff, i);
      } else {
        dequant_dword(dw, tb, bw);
      }
#pragma unroll
      for (int tt = 0; tt < T; ++tt)
        acc[tt][d % G] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
            __builtin_bit_cast(half8v, xa[tt][d / G]),
            __builtin_bit_cast(half8v, u32x4{bw[0], bw[1], bw[2], bw[3]}), acc[tt][d % G], 0, 0,
            0);
    }
    // Lane l holds D[4 (l / 16) + r][l % 16] in component r: D row i is batch row i % MB of
    // dword group i / MB (so lane l's rows belong to group (l / 16) G / 4), column l % 16 the
    // weight row.
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
      float4v mine = acc[tt][0];
#pragma unroll
      for (int s = 1; s < G; ++s)
        if (my_group == s) mine = acc[tt][s];
      s_red[par][w][tt][lane] = mine;
    }
    __syncthreads();
    if (t < NOUT) {
      const int tt = ri / MB, mrow = ri % MB;
      float sum = 0.0f;
#pragma unroll
      for (int s = 0; s < G; ++s) {
        const int i = s * MB + mrow;
        const int l = 16 * (i >> 2) + rj, r = i & 3;
#pragma unroll
        for (int w2 = 0; w2 < WAVES; ++w2) sum += s_red[par][w2][tt][l][r];
      }
#pragma unroll
      for (int h = 0; h < NRES; ++h)
        if (h == held) res[h] = sum * scale;
    }
    par ^= 1;
    ++held;
    blast = b;
    if (held == NRES) flush();
  };
  // Every path through the loop issues the same loads (blocks past the end get size-0
  // descriptors), so the compiler's waits stay exact. The barrier inside block() is reached by
  // the whole workgroup: the loop bounds depend only on the block index.
  for (int b = b0; b < nblocks; b += 2 * gb) {
    load_block(b + gb, q[1]);
    block(b, q[0]);
    load_block(b + 2 * gb, q[0]);
    if (b + gb < nblocks) block(b + gb, q[1]);
  }
  flush();
}

// ------------------------------------------------------------------ split-K MFMA, 8-bit codes
//
// The split-K scheme of k_mfma_sk on one code byte per weight: 16 wavefronts, m <= 16,
// K = 512 ND (ND = 4, 8, 16 MFMAs per lane and block), batch groups G as in k_mfma_sk. Each
// weight is looked up in the LDS table of float16 images (one private copy per lane, 64 KiB,
// two lookups per float16 pair), so the 16 wavefronts' transpose buffers must be small: they
// run in phases of 128 code bytes per row (4 MFMAs) through 2.3 KiB per wavefront. Phase p of a
// block is loaded as two instructions of 8 rows x 128 B, written to the buffer, and the same
// registers are refilled at once with phase p of the workgroup's next block (one block of
// look-ahead in 2 ND / 4 registers). Lane (j, g) then reads row j, bytes [32 g, 32 g + 32) of
// the phase: MFMA d = 4 p + m contracts k = w S + 128 p + 32 g + 8 m + 0..7 (natural order),
// S = 32 ND. One launch serves one linear (its table fills LDS). Measured on MI355X against the
// stepped MFMA kernel (8-bit): 8192 -> 28672 at m = 5 / 8: 57.4 / 57.6 -> 42.1 / 42.5 us,
// 4096 -> 14336 at m = 8: 28.1 -> 14.2 us, 8192 -> 2048 at m = 16: 48.8 -> 17.1 us; but
// 8192 -> 28672 at m = 16: 57.9 -> 60.4 us, so m > 8 at K = 8192 and N > 16384 stays on the
// stepped kernel.
template <int ND, int G>
__global__ __launch_bounds__(1024) void k_mfma_sk8(const uint16_t* __restrict__ x,
                                                   const uint8_t* __restrict__ codes, int n_rows,
                                                   int nblocks, int k_cols, int m_rows,
                                                   float* __restrict__ y, float scale, Lut256 lut) {
  static_assert(ND == 4 || ND == 8 || ND == 16, "K = 512 ND");
  static_assert(G == 1 || G == 2, "batch groups");
  constexpr int W = 16;
  constexpr int NP = ND / 4;             // phases per block
  constexpr int TP = 128 + 16;           // transpose pitch (bytes)
  constexpr int NRES = 4;
  constexpr int MB = 16 / G;
  constexpr int XR = ND / G;
  __shared__ __attribute__((aligned(16))) uint32_t s_lut[kLutWords];
  __shared__ __attribute__((aligned(16))) uint8_t s_ct[W][16 * TP];
  __shared__ __attribute__((aligned(16))) float4v s_red[2][W][64];
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int j = lane & 15, g = lane >> 4;
  const uint32_t laneoff = (uint32_t)lane << 2;
  const int slice0 = w * 32 * ND;        // first weight (and code byte) of this wavefront's slice
  u32x4 xa[XR];
  {
    const int mrow = j % MB, sg = j / MB;
    const bool live = mrow < m_rows;
    const int64_t base = (int64_t)(live ? mrow : 0) * k_cols + slice0 + 32 * g;
#pragma unroll
    for (int r = 0; r < XR; ++r) {
      const int d = G * r + sg;
      const u32x4 v = *reinterpret_cast<const u32x4*>(x + base + 128 * (d >> 2) + 8 * (d & 3));
      xa[r] = live ? v : u32x4{0u, 0u, 0u, 0u};
    }
  }
  auto load_phase = [&](int b, int p, u32x4 (&q)[2]) {
    const int bb = b < nblocks ? b : nblocks - 1;
    const int64_t base = (int64_t)bb * 16 * k_cols;
    const int64_t avail = (int64_t)n_rows * k_cols - base;
    const int size = b < nblocks ? (int)(avail < 16 * (int64_t)k_cols ? avail : 16 * (int64_t)k_cols) : 0;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(codes + base), (short)0, size, kBufferRsrcWord3);
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int off = (8 * c + (lane >> 3)) * k_cols + slice0 + 128 * p + 16 * (lane & 7);
      q[c] = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, kCachePolicyNT);
    }
  };
  const int gb = (int)gridDim.x;
  u32x4 q[NP][2];
#pragma unroll
  for (int p = 0; p < NP; ++p) load_phase(blockIdx.x, p, q[p]);
  fill_single_lut<1024>(s_lut, lut);
  __syncthreads();

  float res[NRES];
  int held = 0, blast = 0, par = 0;
  const int ri = t >> 4, rj = t & 15;
  auto flush = [&]() {
    if (t < 16 * MB && ri < m_rows) {
#pragma unroll
      for (int h = 0; h < NRES; ++h) {
        if (h < held) {
          const int b = blast - (held - 1 - h) * gb;
          const int row = b * 16 + rj;
          if (row < n_rows) y[(int64_t)ri * n_rows + row] = res[h];
        }
      }
    }
    held = 0;
  };
  uint8_t* s_cw = s_ct[w];
  const int my_group = (lane >> 4) * G / 4;
  for (int b = blockIdx.x; b < nblocks; b += gb) {
    float4v acc[G];
#pragma unroll
    for (int s = 0; s < G; ++s) acc[s] = float4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      // LDS operations of one wavefront complete in order: the reads see the writes.
#pragma unroll
      for (int c = 0; c < 2; ++c)
        *reinterpret_cast<u32x4*>(s_cw + (8 * c + (lane >> 3)) * TP + 16 * (lane & 7)) = q[p][c];
      load_phase(b + gb, p, q[p]);
      __builtin_amdgcn_wave_barrier();
      u32x4 o[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        o[i] = *reinterpret_cast<const u32x4*>(s_cw + j * TP + 32 * g + 16 * i);
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const int d = 4 * p + m;
        const u32x4 od = o[m >> 1];
        const uint32_t d0 = (m & 1) ? od.z : od.x;
        const uint32_t d1 = (m & 1) ? od.w : od.y;
        const u32x4 bw{single_pair(s_lut, d0, laneoff, 0), single_pair(s_lut, d0, laneoff, 1),
                       single_pair(s_lut, d1, laneoff, 0), single_pair(s_lut, d1, laneoff, 1)};
        acc[d % G] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
            __builtin_bit_cast(half8v, xa[d / G]), __builtin_bit_cast(half8v, bw), acc[d % G],
            0, 0, 0);
      }
    }
    float4v mine = acc[0];
#pragma unroll
    for (int s = 1; s < G; ++s)
      if (my_group == s) mine = acc[s];
    s_red[par][w][lane] = mine;
    __syncthreads();
    if (t < 16 * MB) {
      float sum = 0.0f;
#pragma unroll
      for (int s = 0; s < G; ++s) {
        const int i = s * MB + ri;
        const int l = 16 * (i >> 2) + rj, r = i & 3;
#pragma unroll
        for (int w2 = 0; w2 < W; ++w2) sum += s_red[par][w2][l][r];
      }
#pragma unroll
      for (int h = 0; h < NRES; ++h)
        if (h == held) res[h] = sum * scale;
    }
    par ^= 1;
    ++held;
    blast = b;
    if (held == NRES) flush();
  }
  flush();
}

// ------------------------------------------------------------------ device fit, exact Eq. 5
//
// One pass of the radix selection described in fit_detail.h. Workgroup g takes the weights
// [g C, (g + 1) C), C = fit_chunk(PASS, n, CUs), and accumulates per bin, in LDS, the count and the
// integer sums of (m^2 >> 24) and (m^2 & 0xFFFFFF) of the weights the pass selects (m = integer
// significand of |w|, m^2 < 2^48). The LDS word a holds count << 44 | sum of (m^2 >> 24): at
// most C <= 2^19 weights per workgroup keep the sum below 2^43 and the count below 2^20, so one
// 64-bit add updates both. Pass 1, which adds every weight, keeps two copies of its bins (even
// and odd lanes), halving the lanes of one instruction that hit the same LDS word; its 64 KiB
// then fit two workgroups per CU, so its chunks are twice as long and the grid runs in one
// round (measured on the 8192 x 28672 weights: the fit 0.868 -> 0.840 ms). Passes 2 and 3 keep
// chunks of 2^18: longer ones halve the bins they flush but leave half the workgroups to
// stream, which measured slower. Non-empty bins are then added to the global bins with 64-bit
// integer atomics, which are exact and independent of order. Pass 1 also takes the largest bit
// pattern and flags NaN / Inf.
constexpr int64_t kFitChunk = int64_t(1) << 18;
constexpr int kFitThreads = 512;
// Largest chunk of a pass: the bound that keeps every LDS word of a workgroup below overflow.
constexpr int64_t fit_chunk_max(int pass) { return pass == 1 ? 2 * kFitChunk : kFitChunk; }
// Chunk of a pass over n weights: the largest chunk, or less for tensors too small to give
// every CU its share (about two workgroups per CU in pass 1, four in passes 2 and 3), in
// multiples of 4096 weights. Measured on MI355X: the 4096 x 1024 projections of a decode layer
// ran pass 1 on 8 workgroups (140 us) with the largest chunk.
int64_t fit_chunk(int pass, int64_t n, int cus) {
  const int64_t target = (int64_t)cus * (pass == 1 ? 2 : 4);
  int64_t c = (n + target - 1) / target;
  c = (c + 4095) / 4096 * 4096;
  return c < fit_chunk_max(pass) ? c : fit_chunk_max(pass);
}

template <int PASS>
__global__ __launch_bounds__(kFitThreads) void k_fit_hist(const float* __restrict__ w, int64_t n,
                                                         int64_t C, uint32_t sel,
                                                         unsigned long long* __restrict__ bins,
                                                         unsigned int* __restrict__ flags) {
  constexpr int NB = PASS == 1 ? logbq_detail::kFitBins1
                     : PASS == 2 ? logbq_detail::kFitBins2 : logbq_detail::kFitBins3;
  constexpr int REP = PASS == 1 ? 2 : 1;
  __shared__ unsigned long long s_a[REP * NB];
  __shared__ unsigned long long s_c[REP * NB];
  __shared__ unsigned int s_max, s_bad;
  const int t = threadIdx.x;
  for (int i = t; i < REP * NB; i += kFitThreads) {
    s_a[i] = 0;
    s_c[i] = 0;
  }
  const int rep = REP == 1 ? 0 : (t & 1) * NB;
  if (t == 0) {
    s_max = 0;
    s_bad = 0;
  }
  __syncthreads();
  uint32_t kmax = 0, bad = 0;
  auto add = [&](uint32_t u) {
    const uint32_t key = u & 0x7FFFFFFFu;
    bool take;
    uint32_t bin;
    if (PASS == 1) {
      kmax = key > kmax ? key : kmax;
      bad |= key >= 0x7F800000u ? 1u : 0u;
      take = true;
      bin = key >> 20;
    } else if (PASS == 2) {
      take = (key >> 20) == sel;
      bin = (key >> 11) & 0x1FFu;
    } else {
      take = (key >> 11) == sel;
      bin = key & 0x7FFu;
    }
    if (take) {
      const uint64_t m = (key & 0x7FFFFFu) | (key >= 0x800000u ? 0x800000u : 0u);
      const uint64_t q = m * m;
      atomicAdd(&s_a[rep + bin], (1ull << 44) | (q >> 24));
      atomicAdd(&s_c[rep + bin], (unsigned long long)(q & 0xFFFFFFu));
    }
  };
  const int64_t begin = (int64_t)blockIdx.x * C;   // C <= fit_chunk_max(PASS), a multiple of 4
  const int64_t end = n - begin < C ? n : begin + C;
  const int64_t vend = begin + ((end - begin) & ~int64_t(3));
  // Passes 1 and 2 take U = 4 vectors per thread per iteration, all requested before any is
  // binned (pass 1 waits on its LDS atomics, and with two workgroups per CU one vector in
  // flight per thread left HBM idle: 263 -> 244 us and 196 -> 182 us per pass on the
  // 8192 x 28672 tensor, MI355X); pass 3 bins almost nothing and streams best with U = 1.
  constexpr int U = PASS == 3 ? 1 : 4;
  for (int64_t i0 = begin + 4 * t; i0 < vend; i0 += 4 * kFitThreads * U) {
    u32x4 v[U];
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int64_t i = i0 + (int64_t)j * 4 * kFitThreads;
      v[j] = i < vend ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(w + i))
                      : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int j = 0; j < U; ++j) {
      if (i0 + (int64_t)j * 4 * kFitThreads < vend) {
        add(v[j].x);
        add(v[j].y);
        add(v[j].z);
        add(v[j].w);
      }
    }
  }
  if (vend + t < end) add(__float_as_uint(w[vend + t]));
  if (PASS == 1) {
    atomicMax(&s_max, kmax);
    if (bad) atomicOr(&s_bad, 1u);
  }
  __syncthreads();
  for (int i = t; i < NB; i += kFitThreads) {
    unsigned long long cnt = 0, hi = 0, lo = 0;
    for (int r = 0; r < REP; ++r) {
      const unsigned long long a = s_a[r * NB + i];
      cnt += a >> 44;
      hi += a & ((1ull << 44) - 1);
      lo += s_c[r * NB + i];
    }
    if (cnt == 0) continue;
    atomicAdd(&bins[3 * i], cnt);
    atomicAdd(&bins[3 * i + 1], hi);
    atomicAdd(&bins[3 * i + 2], lo);
  }
  if (PASS == 1 && t == 0) {
    atomicMax(&flags[0], s_max);
    if (s_bad) atomicOr(&flags[1], 1u);
  }
}

__global__ void k_fill_u64(unsigned long long* __restrict__ p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

// ------------------------------------------------------------------ host helpers

// IEEE binary32 -> binary16, round to nearest even.
uint16_t f32_to_f16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  const uint32_t sign = (u >> 16) & 0x8000u;
  const uint32_t e = (u >> 23) & 0xFFu;
  uint32_t m = u & 0x7FFFFFu;
  if (e == 0xFF) return (uint16_t)(sign | 0x7C00u | (m ? 0x200u : 0u));
  const int32_t ee = (int32_t)e - 127 + 15;
  if (ee >= 31) return (uint16_t)(sign | 0x7C00u);
  if (ee <= 0) {
    if (ee < -10) return (uint16_t)sign;
    m |= 0x800000u;
    const int shift = 14 - ee;
    uint32_t hm = m >> shift;
    const uint32_t rem = m & ((1u << shift) - 1u);
    const uint32_t halfway = 1u << (shift - 1);
    if (rem > halfway || (rem == halfway && (hm & 1u))) ++hm;
    return (uint16_t)(sign | hm);
  }
  uint32_t hm = m >> 13;
  const uint32_t rem = m & 0x1FFFu;
  uint32_t out = sign | ((uint32_t)ee << 10) | hm;
  if (rem > 0x1000u || (rem == 0x1000u && (hm & 1u))) ++out;
  return (uint16_t)out;
}

// float16 image of a codebook: lut16 = f16(cb / 2^e), scale = 2^e.
// float16 image of a 2^BITS-entry codebook, scaled by 2^-e so that the largest magnitude lies
// in [2^14, 2^15); *scale = 2^e multiplies the results back (exactly).
template <int BITS>
void make_lut(const float* cb, typename LutOf<BITS>::type* lut, float* scale) {
  constexpr int kN = 1 << BITS;
  float mx = 0.0f;
  for (int i = 0; i < kN; ++i) mx = std::fmax(mx, std::fabs(cb[i]));
  int e = 0;
  if (mx > 0.0f) {
    int E;
    std::frexp(mx, &E);          // mx = f * 2^E, f in [0.5, 1)
    e = E - 15;                  // mx / 2^e in [2^14, 2^15)
  }
  for (int i = 0; i < kN / 2; ++i)
    lut->h[i] = (uint32_t)f32_to_f16(std::ldexp(cb[2 * i], -e)) |
                ((uint32_t)f32_to_f16(std::ldexp(cb[2 * i + 1], -e)) << 16);
  *scale = std::ldexp(1.0f, e);
}

void make_lut16(const float* cb, Lut16* lut, float* scale) { make_lut<4>(cb, lut, scale); }

struct DeviceInfo { int cus = 0; };

int device_cus() {
  static std::mutex mu;
  static DeviceInfo info[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  std::lock_guard<std::mutex> lock(mu);
  if (info[dev].cus == 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    info[dev].cus = cus;
  }
  return info[dev].cus;
}

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int32_t launch_status() {
  return hipGetLastError() == hipSuccess ? LOGBQ_OK : LOGBQ_ERR_HIP;
}

int64_t grid_for(int64_t items, int64_t per_block, int64_t cap) {
  int64_t g = (items + per_block - 1) / per_block;
  if (g > cap) g = cap;
  if (g < 1) g = 1;
  return g;
}

// Zeroes y[0 .. count) on the stream (one 16-byte store per thread and pass).
void fill_zero(float* y, int64_t count, int cus, hipStream_t st) {
  hipLaunchKernelGGL(k_fill_zero, dim3((unsigned)grid_for((count + 3) / 4, 256, (int64_t)cus * 4)),
                     dim3(256), 0, st, y, count);
}

template <int BITS, int M, int CPL>
void launch_gemv(int grid, hipStream_t st, const uint16_t* x, int k, int wk, int stage_x,
                 const GemvSegs<BITS>& segs) {
  constexpr int NBUF = (CPL <= 2 && M <= 2) ? 3 : 2;
  if (wk == 1)
    hipLaunchKernelGGL((k_gemv<BITS, M, CPL, false, NBUF>), dim3((unsigned)grid), dim3(512), 0,
                       st, x, segs.s[0].codes, k, segs.s[0].n_rows, segs.count, 1, stage_x, segs);
  else
    hipLaunchKernelGGL((k_gemv<BITS, M, CPL, true, NBUF>), dim3((unsigned)grid), dim3(512), 0,
                       st, x, segs.s[0].codes, k, segs.s[0].n_rows, segs.count, wk, stage_x, segs);
}

template <int BITS>
bool dispatch_gemv(int m, int cpl, int grid, hipStream_t st, const uint16_t* x, int k, int wk,
                   int stage_x, const GemvSegs<BITS>& segs) {
#define LOGBQ_G(MM, CC) \
  if (m == MM && cpl == CC) { launch_gemv<BITS, MM, CC>(grid, st, x, k, wk, stage_x, segs); return true; }
  LOGBQ_G(1, 1) LOGBQ_G(1, 2) LOGBQ_G(1, 3) LOGBQ_G(1, 4) LOGBQ_G(1, 5) LOGBQ_G(1, 6) LOGBQ_G(1, 7) LOGBQ_G(1, 8)
  LOGBQ_G(2, 1) LOGBQ_G(2, 2) LOGBQ_G(2, 3) LOGBQ_G(2, 4)
  LOGBQ_G(3, 1) LOGBQ_G(3, 2)
  LOGBQ_G(4, 1) LOGBQ_G(4, 2)
  LOGBQ_G(5, 1) LOGBQ_G(6, 1) LOGBQ_G(7, 1) LOGBQ_G(8, 1)
#undef LOGBQ_G
  return false;
}

// GEMV configuration for m batch rows and k columns of BITS-bit codes: WK wavefronts per row
// and CPL 16-byte code chunks per lane, keeping at most 8 / m chunks of activations per lane.
// Returns false when even WK = 8 does not fit (the MFMA path takes those shapes).
template <int BITS>
bool gemv_config(int m, int k, int* wk, int* cpl) {
  if (m < 1 || m > 8) return false;
  const int nchunks = k / kChunkW<BITS>;
  const int cplmax = 8 / m;
  for (int w = 1; w <= 8; w *= 2) {
    const int per = (nchunks + 64 * w - 1) / (64 * w);
    // The split-row 4-bit kernels keep at most 7 chunks per lane (8 would spill registers).
    const int cap = (w == 1 || cplmax < 7 || BITS == 8) ? cplmax : 7;
    if (per <= cap && (w == 1 || nchunks >= 32 * w)) {
      *wk = w;
      *cpl = per < 1 ? 1 : per;
      return true;
    }
  }
  return false;
}

// The configuration one linear of n rows takes. At one batch row, the long rows of a narrow
// 4-bit linear stream faster with two wavefronts per row (measured on MI355X: n = 4096,
// k = 14336: 7.96 -> 7.46 us; n = 2048, k = 8192: 4.42 -> 4.14 us). Wider linears and shorter
// rows were slower with two or four (e.g. n = 28672, k = 8192: 19.7 -> 20.1 us; n = 4096,
// k = 4096: 4.0 -> 4.8 us).
template <int BITS>
bool gemv_config_rows(int m, int k, int64_t n, int* wk, int* cpl) {
  if (!gemv_config<BITS>(m, k, wk, cpl)) return false;
  const int nchunks = k / kChunkW<BITS>;
  if (BITS == 4 && m == 1 && *wk == 1 && n <= 4096 && nchunks >= 256) {
    const int per = (nchunks + 127) / 128;
    if (per <= 7) {
      *wk = 2;
      *cpl = per;
    }
  }
  return true;
}

struct LinearJob {
  const uint8_t* codes;
  int64_t n;
  const float* codebook;
  float* y;
};

int32_t validate_job(const LinearJob& j, int64_t m, int64_t k, int entries = 16) {
  if (!j.codebook || j.n < 0) return LOGBQ_ERR_INVALID_ARG;
  if (j.n > INT32_MAX) return LOGBQ_ERR_UNSUPPORTED;
  for (int i = 0; i < entries; ++i)
    if (!std::isfinite(j.codebook[i])) return LOGBQ_ERR_INVALID_ARG;
  if (m == 0 || j.n == 0) return LOGBQ_OK;
  if (!j.y) return LOGBQ_ERR_INVALID_ARG;
  if (!aligned16(j.y)) return LOGBQ_ERR_UNSUPPORTED;
  if (k > 0) {
    if (!j.codes) return LOGBQ_ERR_INVALID_ARG;
    if (!aligned16(j.codes)) return LOGBQ_ERR_UNSUPPORTED;
  }
  return LOGBQ_OK;
}

// float16 byte tables for the register dequant; false unless the codebook is sign-symmetric
// with a non-negative positive half (every fitted codebook is).
bool make_lut_bytes(const float* cb, LutBytes* tb, float* scale) {
  for (int k = 0; k < 8; ++k)
    if (!(cb[k] >= 0.0f)) return false;
  if (cb[8] != 0.0f) return false;
  for (int k = 1; k < 8; ++k)
    if (cb[8 + k] != -cb[k]) return false;
  Lut16 lut;
  make_lut16(cb, &lut, scale);
  uint32_t lo[2] = {0, 0}, hi[2] = {0, 0};
  for (int k = 0; k < 8; ++k) {
    const uint32_t h16 = (lut.h[k >> 1] >> (16 * (k & 1))) & 0xFFFFu;
    lo[k >> 2] |= (h16 & 0xFFu) << (8 * (k & 3));
    hi[k >> 2] |= (h16 >> 8) << (8 * (k & 3));
  }
  tb->lo0 = lo[0]; tb->lo1 = lo[1]; tb->hi0 = hi[0]; tb->hi1 = hi[1];
  return true;
}

// Largest batch: the MFMA grid's y dimension (at most 65535) covers 64 batch rows or more each.
constexpr int64_t kMaxBatchRows = 65535LL * 64;

// The stepped kernel with 64-row workgroups (k_mfma2_narrow) runs when its whole grid fits on
// the chip at once, one workgroup per CU (gfx950: 256 CUs; a fixed count keeps the path choice
// a function of m, k and N alone). There each CU walks K for 64 rows instead of 128 (or for
// none, when the 128-row grid leaves it idle). Measured on MI355X (graph replay, codes
// streamed from HBM), 64-row against 128-row workgroups, bit-identical results (each output is
// the same K walk): register tables 0.73-0.89 of the time for N = 2048 .. 16384,
// K = 2048 .. 14336, m = 9 .. 96 (e.g. 4096 x 4096 at m = 64: 26.6 -> 20.9 us, 4096 -> 14336 at
// m = 96: 37.9 -> 29.6 us); the LDS tables (8-bit codes, other codebooks) 0.66-0.81 (8-bit
// 4096 x 4096 at m = 48: 40.9 -> 27.0 us, 8192 x 8192 at m = 64: 86.0 -> 59.1 us; 4-bit
// 4096 x 4096 at m = 64: 30.1 -> 21.0 us); at N = 28672 (448 workgroups) 1.04-1.44 times the
// time. `cap` is the kernel's batch tiles per workgroup column (8 with register tables, 4 with
// the LDS table). This rule now decides between the stepped and the K-quartered kernel, and is
// what step_config below falls back to where no launch shape fits on the chip.
constexpr int64_t kNarrowMaxWorkgroups = 256;
bool narrow_fits(int M, int64_t N, int cap = 8) {
  const int64_t gy = M > 16 * cap ? (M + 16 * cap - 1) / (16 * cap) : 1;
  return ((N + 63) / 64) * gy <= kNarrowMaxWorkgroups;
}

// Launch shape of the stepped kernel: 64-row (narrow) or 128-row workgroups, batch tiles of 16
// rows per workgroup column, and K in one or two parts (two: the output is zeroed first and each
// part adds into it).
struct StepCfg {
  bool narrow;
  int mt16;
  int ks;
};
// The shape is the cheapest, by a cost model, of every shape whose grid fits on the chip at
// once (at most one workgroup per CU): 64 or 128 rows, t = t0, t0 / 2, ... 1 batch tiles
// (halving rounds up; t0 = ceil(m / 16) up to the cap: 8 with register tables, 4 with the LDS
// table), one K part, or two when K has at least 16 steps of 256. A workgroup's time is its
// steps times a per-step time that grows with t (activation staging, MFMAs and LDS reads) on
// top of a fixed part (code loads and dequantization); two K parts add a fixed cost (the
// zeroing launch, the atomic adds, a shorter pipeline). The constants are least-squares fits to
// MI355X measurements (graph replay, codes streamed from HBM) of 64- and 128-row workgroups at
// every t on 4096 x 14336, 4096 x 4096, 14336 x 4096 and 2048 x 8192 (plus 1024 x 4096 for
// register tables), one set per kind of dequantization. Against 64-row workgroups with all t0
// tiles and one K part (the rule above), e.g.: 4096 x 14336 at m = 128, register tables
// (128 rows, t = 2, two parts) 109.9 -> 35.9 us; at m = 64, 8-bit codes (64 rows, t = 2, two
// parts) 93.1 -> 34.4 us; 2048 x 8192 at m = 64, a 4-bit LDS table (64 rows, t = 1, two parts)
// 38.4 -> 13.5 us; 14336 x 4096 at m = 128, register tables (128 rows, t = 4, one part)
// 37.2 -> 30.3 us. Where no shape fits (N = 28672) the rule above stands.
struct StepCosts {
  double fixed64, tile64, fixed128, tile128, two_parts;   // us per step of 256; us
};
constexpr StepCosts kCostsRegister = {0.376, 0.184, 0.500, 0.300, 5.0};
constexpr StepCosts kCostsTable4 = {0.283, 0.198, 0.205, 0.374, 3.1};
constexpr StepCosts kCostsTable8 = {0.422, 0.279, 0.156, 0.600, 3.0};
StepCfg step_config(int M, int64_t N, int K, int bits, bool symmetric) {
  const bool reg = bits == 4 && symmetric;
  const int cap = reg ? 8 : 4;
  int t0 = (M + 15) / 16;
  if (t0 > cap) t0 = cap;
  StepCfg best{narrow_fits(M, N, cap), t0, 1};
  const StepCosts& cc = reg ? kCostsRegister : bits == 4 ? kCostsTable4 : kCostsTable8;
  const int64_t nsteps = ((int64_t)K + kM2Step - 1) / kM2Step;
  double best_cost = -1.0;
  for (int rows = 128; rows >= 64; rows /= 2)
    for (int mt = t0;; mt = (mt + 1) / 2) {
      // 8-bit codes in 128-row workgroups with one batch tile take far longer than the linear
      // fit says (4096 -> 14336 at m = 128: 73.4 us, against 48.7 with two tiles and two K
      // parts); those shapes are left out.
      for (int ks = 1; ks <= (nsteps >= 16 ? 2 : 1) && !(bits == 8 && rows == 128 && mt == 1);
           ++ks) {
        const int64_t wgs = ((N + rows - 1) / rows) * ((M + 16 * mt - 1) / (16 * mt)) * ks;
        if (wgs > kNarrowMaxWorkgroups) continue;
        const double per_step = rows == 128 ? cc.fixed128 + mt * cc.tile128
                                            : cc.fixed64 + mt * cc.tile64;
        const double cost = (double)((nsteps + ks - 1) / ks) * per_step +
                            (ks == 2 ? cc.two_parts : 0.0);
        if (best_cost < 0.0 || cost < best_cost) {
          best_cost = cost;
          best = {rows == 64, mt, ks};
        }
      }
      if (mt == 1) break;
    }
  return best;
}

template <int BITS>
int32_t launch_mfma(const uint16_t* x, int M, int K, const LinearJob& j, hipStream_t st) {
  const int N = (int)j.n;
  // The kernel reads a workgroup's 128 rows through one buffer descriptor of at most 2^31 bytes.
  if ((int64_t)128 * K * BITS / 8 >= ((int64_t)1 << 31)) return LOGBQ_ERR_UNSUPPORTED;
  LutBytes tb = {0, 0, 0, 0};
  typename LutOf<BITS>::type lut;
  float scale;
  // 4-bit codes: register dequantization needs a sign-symmetric codebook (every fitted one
  // is); any other codebook, and every 8-bit one, uses the LDS table with at most 4 batch tiles
  // per workgroup column.
  const bool symmetric = BITS == 4 && make_lut_bytes(j.codebook, &tb, &scale);
  make_lut<BITS>(j.codebook, &lut, &scale);
  // Batch tiles of 16 rows: up to 8 per workgroup column (128 rows). Up to 4 tiles use the
  // LDS table; more tiles leave LDS to the activation ring and dequantize in registers.
  const StepCfg cfg = step_config(M, N, K, BITS, symmetric);
  const int mt16 = cfg.mt16;
  const bool narrow = cfg.narrow;
  const int rows_wg = narrow ? 64 : 128;
  dim3 grid((unsigned)((N + rows_wg - 1) / rows_wg),
            (unsigned)((M + 16 * mt16 - 1) / (16 * mt16)), (unsigned)cfg.ks);
  if (cfg.ks > 1) {
    const int cus = device_cus();
    if (cus <= 0) return LOGBQ_ERR_HIP;
    fill_zero(j.y, (int64_t)M * N, cus, st);
  }
#define LOGBQ_M2(MT, ST, PR) hipLaunchKernelGGL((k_mfma2<BITS, MT, ST, PR, (MT <= 2)>), grid, dim3(512), 0, st, j.codes, x, j.y, N, K, M, tb, lut, scale)
#define LOGBQ_M2N(MT, PR) hipLaunchKernelGGL((k_mfma2_narrow<BITS, MT, PR, (MT <= 2)>), grid, dim3(256), 0, st, j.codes, x, j.y, N, K, M, tb, lut, scale)
  if constexpr (BITS == 4) {
    // Register dequantization whenever the codebook allows it: measured 1 to 2.5 us faster than
    // the LDS table at m = 4 .. 32 on the 8192 x 28672 layer, with bit-identical results.
    if (narrow && symmetric) {
      switch (mt16) {
        case 1: LOGBQ_M2N(1, false); break;
        case 2: LOGBQ_M2N(2, false); break;
        case 3: LOGBQ_M2N(3, false); break;
        case 4: LOGBQ_M2N(4, false); break;
        case 5: LOGBQ_M2N(5, false); break;
        case 6: LOGBQ_M2N(6, false); break;
        case 7: LOGBQ_M2N(7, false); break;
        default: LOGBQ_M2N(8, false); break;
      }
    } else if (narrow) {
      switch (mt16) {
        case 1: LOGBQ_M2N(1, true); break;
        case 2: LOGBQ_M2N(2, true); break;
        case 3: LOGBQ_M2N(3, true); break;
        default: LOGBQ_M2N(4, true); break;
      }
    } else if (symmetric) {
      switch (mt16) {
        case 1: LOGBQ_M2(1, 4, false); break;
        case 2: LOGBQ_M2(2, 4, false); break;
        case 3: LOGBQ_M2(3, 4, false); break;
        case 4: LOGBQ_M2(4, 4, false); break;
        case 5: LOGBQ_M2(5, 4, false); break;
        case 6: LOGBQ_M2(6, 4, false); break;
        case 7: LOGBQ_M2(7, 4, false); break;
        default: LOGBQ_M2(8, 4, false); break;
      }
    } else {
      switch (mt16) {
        case 1: LOGBQ_M2(1, 4, true); break;
        case 2: LOGBQ_M2(2, 4, true); break;
        case 3: LOGBQ_M2(3, 4, true); break;
        default: LOGBQ_M2(4, 4, true); break;
      }
    }
  } else if (narrow) {
    switch (mt16) {
      case 1: LOGBQ_M2N(1, true); break;
      case 2: LOGBQ_M2N(2, true); break;
      case 3: LOGBQ_M2N(3, true); break;
      default: LOGBQ_M2N(4, true); break;
    }
  } else {
    switch (mt16) {
      case 1: LOGBQ_M2(1, 4, true); break;
      case 2: LOGBQ_M2(2, 4, true); break;
      case 3: LOGBQ_M2(3, 4, true); break;
      default: LOGBQ_M2(4, 4, true); break;
    }
  }
#undef LOGBQ_M2
#undef LOGBQ_M2N
  return launch_status();
}

// Split-K launch on 8-bit codes (one linear per launch).
bool sk8_shape(int M, int K) { return M >= 2 && M <= 16 && (K == 2048 || K == 4096 || K == 8192); }

int32_t launch_sk8(const uint16_t* x, int M, int K, const LinearJob& j, hipStream_t st, int cus) {
  Lut256 lut;
  float scale;
  make_lut<8>(j.codebook, &lut, &scale);
  const int nblocks = (int)((j.n + 15) / 16);
  const int grid = nblocks < cus ? nblocks : cus;
  const bool g2 = M <= 8;
#define LOGBQ_SK8(ND, GG)                                                                        \
  hipLaunchKernelGGL((k_mfma_sk8<ND, GG>), dim3((unsigned)grid), dim3(1024), 0, st, x, j.codes, \
                     (int)j.n, nblocks, K, M, j.y, scale, lut)
  switch (K) {
    case 2048: if (g2) LOGBQ_SK8(4, 2); else LOGBQ_SK8(4, 1); break;
    case 4096: if (g2) LOGBQ_SK8(8, 2); else LOGBQ_SK8(8, 1); break;
    default: if (g2) LOGBQ_SK8(16, 2); else LOGBQ_SK8(16, 1); break;
  }
#undef LOGBQ_SK8
  return launch_status();
}

// K-quartered MFMA path on 8-bit codes: m > 64 at N >= 16384.
// (K < 2^24 keeps the 128-row buffer descriptor below 2^31 bytes.)
bool kq8_shape(int M, int64_t N, int K) { return M > 64 && N >= 16384 && K < (1 << 24); }

int32_t launch_kq8(const uint16_t* x, int M, int K, const LinearJob& j, hipStream_t st) {
  Lut256 lut;
  float scale;
  make_lut<8>(j.codebook, &lut, &scale);
  const int N = (int)j.n;
  dim3 grid((unsigned)((N + 127) / 128), (unsigned)((M + 127) / 128));
  hipLaunchKernelGGL(k_mfma_kq8, grid, dim3(512), 0, st, j.codes, x, j.y, N, K, M, scale, lut);
  return launch_status();
}

// K-quartered MFMA path (4-bit, sign-symmetric codebooks): m > 96 at N >= 4096.
// (K < 2^25 keeps the 128-row buffer descriptor below 2^31 bytes.)
bool kq_shape(int M, int64_t N, int K) { return M > 96 && N >= 4096 && K < (1 << 25); }

int32_t launch_kq(const uint16_t* x, int M, int K, const LinearJob& j, hipStream_t st) {
  const int N = (int)j.n;
  LutBytes tb = {0, 0, 0, 0};
  float scale;
  if (!make_lut_bytes(j.codebook, &tb, &scale)) return launch_mfma<4>(x, M, K, j, st);
  dim3 grid((unsigned)((N + 127) / 128), (unsigned)((M + 127) / 128));
  hipLaunchKernelGGL(k_mfma_kq, grid, dim3(512), 0, st, j.codes, x, j.y, N, K, M, tb, scale);
  return launch_status();
}

// Split-K MFMA path: 4-bit codes, 2 <= m <= 32 at K in {1024, 2048, 4096, 8192}, and
// 2 <= m <= 16 at K = 14336 (the down projection of the 8B-shaped decoder). Above m = 16 at
// K = 14336 the stepped kernel in its cost-model shape is faster than split-K launches of at
// most 16 batch rows each (4096 rows at m = 17 / 24 / 32 / 48: 26.4 / 28.7 / 31.4 / 46.6 ->
// 21.0 / 21.0 / 21.0 / 27.2 us on MI355X); at the other K, split-K stays ahead to m = 24 and
// even at m = 32 (e.g. 4096 x 4096 at m = 17: 9.0 vs 11.3 us).
bool sk_shape(int M, int K) {
  return M >= 2 && ((M <= 32 && (K == 1024 || K == 2048 || K == 4096 || K == 8192)) ||
                    (M <= 16 && K == 14336));
}

// Split-K configuration: code dwords per lane and row, wavefronts per workgroup, batch groups,
// batch tiles and K parts (workgroups per block).
struct SkConfig {
  int nd, waves, groups, tiles, kparts;
  bool operator==(const SkConfig& o) const {
    return nd == o.nd && waves == o.waves && groups == o.groups && tiles == o.tiles &&
           kparts == o.kparts;
  }
};
// The configuration of one linear of `blocks` 16-row blocks. It depends only on (m, K, blocks)
// and the codebook's kind, so a grouped launch only joins linears of equal configuration and
// each computes as in a call of its own.
SkConfig sk_config(int M, int K, bool pairs, int blocks) {
  // K = 14336 = 2 x 14 x 512: workgroup pairs of 14 wavefronts, one K half each.
  if (K == 14336) return {16, 14, M <= 8 ? 2 : 1, 1, 2};
  if (M > 16) {   // two batch tiles (register tables only); K = 8192 over workgroup pairs
    const int waves = K >= 2048 ? 16 : 8;
    const int kparts = K == 8192 ? 2 : 1;
    return {K / (32 * waves * kparts), waves, 1, 2, kparts};
  }
  // Narrow layers: one workgroup per block leaves CUs idle, and above m = 8 a lane's
  // activations for all of K take 64 VGPRs; there the K halves go to workgroup pairs
  // (ND = K / 1024). Measured on MI355X (graph replay, codes streamed from HBM), K = 8192:
  // N = 2048 at m = 4 / 8 / 16: 7.27 / 8.52 / 12.52 -> 6.79 / 7.23 / 9.17 us; N = 8192 at
  // m = 12 / 16: 14.32 / 15.80 -> 13.74 / 14.60 us; slower at m <= 8 from N = 3072 on (mixed
  // to N = 6144) and at N >= 14336. K = 4096 gains only above m = 12 at N <= 2048 (N = 1024 at
  // m = 16: 7.08 -> 6.41 us).
  if (!pairs && ((K == 8192 && blocks <= (M <= 8 ? 128 : 512)) ||
                 (K == 4096 && M > 12 && blocks <= 128)))
    return {K / 1024, 16, M <= 8 ? 2 : 1, 1, 2};
  const int waves = (!pairs && K >= 4096) ? 16 : 8;
  return {K / (32 * waves), waves, (!pairs && M <= 8) ? 2 : 1, 1, 1};
}

// Split-K launches for the linears jobs[idx[0..count)] of one call: when every codebook is
// sign-symmetric (register dequantization), one grouped launch per distinct configuration,
// otherwise one launch per linear (above m = 16, and at K = 14336, a codebook that is not
// sign-symmetric takes the stepped MFMA kernel). At K = 14336, m <= 16.
int32_t launch_sk(const uint16_t* x, int M, int K, const LinearJob* jobs, const int* idx,
                  int count, hipStream_t st, int cus) {
  SkSegs segs;
  std::memset(&segs, 0, sizeof(segs));
  Lut16 lut;
  bool all_symmetric = true;
  int total = 0;
  for (int a = 0; a < count; ++a) {
    const LinearJob& j = jobs[idx[a]];
    SkSeg& sg = segs.s[a];
    sg.codes = j.codes;
    sg.y = j.y;
    sg.n_rows = (int)j.n;
    sg.blk_begin = total;
    all_symmetric = make_lut_bytes(j.codebook, &sg.tb, &sg.scale) && all_symmetric;
    total += (int)((j.n + 15) / 16);
  }
  auto launch = [&](int nseg, const SkSegs& sgs, int nblocks, bool pairs, const Lut16& l,
                    const SkConfig& c) -> int32_t {
    // One workgroup per CU (the grid walks the blocks); with two K parts an even grid of
    // workgroup pairs, after zeroing every output the atomic adds will land on.
    int grid = nblocks * c.kparts < cus ? nblocks * c.kparts : cus;
    grid -= grid % c.kparts;
    if (c.kparts == 2)
      for (int a = 0; a < nseg; ++a) fill_zero(sgs.s[a].y, (int64_t)M * sgs.s[a].n_rows, cus, st);
#define LOGBQ_SK(ND, W, GG, TT, KP, PR)                                                          \
  if (c.nd == ND && c.waves == W && c.groups == GG && c.tiles == TT && c.kparts == KP &&         \
      pairs == PR) {                                                                             \
    hipLaunchKernelGGL((k_mfma_sk<ND, W, GG, TT, KP, PR>), dim3((unsigned)grid), dim3(64 * W), 0, \
                       st, x, sgs.s[0].codes, sgs.s[0].n_rows, nseg, nblocks, K, M, sgs, l);     \
    return launch_status();                                                                      \
  }
    LOGBQ_SK(4, 8, 1, 1, 1, true) LOGBQ_SK(8, 8, 1, 1, 1, true)
    LOGBQ_SK(16, 8, 1, 1, 1, true) LOGBQ_SK(32, 8, 1, 1, 1, true)
    LOGBQ_SK(4, 8, 1, 1, 1, false) LOGBQ_SK(4, 8, 2, 1, 1, false)
    LOGBQ_SK(8, 8, 1, 1, 1, false) LOGBQ_SK(8, 8, 2, 1, 1, false)
    LOGBQ_SK(8, 16, 1, 1, 1, false) LOGBQ_SK(8, 16, 2, 1, 1, false)
    LOGBQ_SK(16, 16, 1, 1, 1, false) LOGBQ_SK(16, 16, 2, 1, 1, false)
    LOGBQ_SK(4, 8, 1, 2, 1, false) LOGBQ_SK(4, 16, 1, 2, 1, false)
    LOGBQ_SK(8, 16, 1, 2, 1, false) LOGBQ_SK(8, 16, 1, 2, 2, false)
    LOGBQ_SK(16, 14, 2, 1, 2, false) LOGBQ_SK(16, 14, 1, 1, 2, false)
    LOGBQ_SK(8, 16, 2, 1, 2, false)
    LOGBQ_SK(8, 16, 1, 1, 2, false) LOGBQ_SK(4, 16, 1, 1, 2, false)
#undef LOGBQ_SK
    return LOGBQ_ERR_UNSUPPORTED;
  };
  if (all_symmetric) {
    SkConfig cfg[kMaxSegs];
    bool done[kMaxSegs] = {};
    for (int a = 0; a < count; ++a)
      cfg[a] = sk_config(M, K, false, (int)((jobs[idx[a]].n + 15) / 16));
    for (int a0 = 0; a0 < count; ++a0) {
      if (done[a0]) continue;
      SkSegs grp;
      std::memset(&grp, 0, sizeof(grp));
      int nseg = 0, blocks = 0;
      for (int a = a0; a < count; ++a)
        if (!done[a] && cfg[a] == cfg[a0]) {
          grp.s[nseg] = segs.s[a];
          grp.s[nseg].blk_begin = blocks;
          blocks += (int)((jobs[idx[a]].n + 15) / 16);
          ++nseg;
          done[a] = true;
        }
      const int32_t r = launch(nseg, grp, blocks, false, lut, cfg[a0]);
      if (r != LOGBQ_OK) return r;
    }
    return LOGBQ_OK;
  }
  for (int a = 0; a < count; ++a) {
    const LinearJob& j = jobs[idx[a]];
    SkSegs one;
    std::memset(&one, 0, sizeof(one));
    one.s[0] = segs.s[a];
    one.s[0].blk_begin = 0;
    // Register dequantization for a sign-symmetric codebook (every fitted one), the LDS pair
    // table for any other.
    const bool symmetric = make_lut_bytes(j.codebook, &one.s[0].tb, &one.s[0].scale);
    make_lut16(j.codebook, &lut, &one.s[0].scale);
    const int blocks = (int)((j.n + 15) / 16);
    const int32_t r = ((M > 16 || K == 14336) && !symmetric)
                          ? launch_mfma<4>(x, M, K, j, st)
                          : launch(1, one, blocks, !symmetric, lut,
                                   sk_config(M, K, !symmetric, blocks));
    if (r != LOGBQ_OK) return r;
  }
  return LOGBQ_OK;
}

// Path choice per linear (measured on MI355X). The GEMV's time grows with m * N * K (its
// products are VALU dot2 per weight and batch row); the MFMA kernel's is about flat in m up to
// 16 but uses only N / 128 workgroups. Measured crossover: the MFMA kernel wins once m >= 3 and
// m * N > 65536 (N = 28672 from m = 3, N = 14336 from m = 5; at N = 8192, m = 8 the GEMV is
// still 1 us faster); the GEMV takes everything else up to m = 8. At 8 bits the stepped MFMA
// kernel looks up every weight in its LDS table and the GEMV stays ahead to m = 4 on every
// layer (8192 -> 28672 at m = 3 / 4: 48.0 / 56.1 us vs 57.2 / 57.3 us; at m = 6: 103 vs 57 us). The choice depends only on
// (m, k, N), so every linear of a grouped call runs the kernel that a single call would run,
// with the same result bits.
//
// Above m = 96 at N >= 4096 the K-quartered kernel replaces the stepped one for 4-bit codes with
// sign-symmetric codebooks (7-11 % faster on the 8192 x 28672 and 4096 x 14336 layers; slower
// on narrow layers, which have too few 128-row workgroups), except where the stepped kernel's
// 64-row grid fits on the chip: there that one is faster (measured at m = 97 .. 256,
// N = 4096 .. 16384, K = 2048 .. 14336: 0.77-1.00 of the K-quartered kernel's time, e.g.
// 4096 x 4096 at m = 128: 37.1 -> 34.3 us, 2048 -> 4096 at m = 128: 23.1 -> 19.3 us).
//
// Where the split-K MFMA kernel applies (4-bit codes, 2 <= m <= 32, K = 1, 2, 4 or 8 Ki), it
// takes 5 <= m <= 16, m = 4 unless N <= 1024 at K = 8192, m = 3 at N >= 4096, and
// 17 <= m <= 32 except m > 20 at K = 8192 and N > 16384. Measured with forced paths over
// N = 1024 .. 28672 and K = 2048 .. 8192: at m = 4 it beats the GEMV except at N = 1024,
// K = 8192 (7.0 vs 6.9 us), e.g. 4096 x 4096: 4.9 vs 5.7 us, 8192 -> 28672: 26.4 vs 37.7 us; at
// m = 3 from N = 4096 (one exception, 4096 -> 6144: 6.2 vs 5.9 us); at m = 2 the GEMV wins
// (8192 -> 28672: 21.9 vs 25.4 us). Up to m = 16 it beats the stepped MFMA kernel on every
// layer (8192 -> 28672 at m = 16: 30.6 vs 31.6 us); at m = 32 on every layer but the widest:
// 4096 x 4096 11.1 vs 20.4 us, 4096 -> 14336 16.7 vs 21.1 us, 8192 -> 2048 13.2 vs 37.5 us,
// 8192 -> 14336 28.6 vs 39.1 us, but 8192 -> 28672 44.4 vs 41.3 us (there it wins to m = 20:
// 38.6 vs 41.0 us).
//
// 8-bit codes take their split-K kernel for 5 <= m <= 8 unless N <= 1024 at K >= 4096, for
// m = 3, 4 at N >= 8192 and for 9 <= m <= 16 unless N > 16384 at K = 8192 (forced-path builds
// over N = 1024 .. 28672, K = 2048 .. 8192: e.g. 4096 x 4096 at m = 8: 7.3 us vs 12.9 us for the
// GEMV; 8192 -> 28672 at m = 5: 40.9 vs 90.7 us; N = 1024, K = 8192 at m = 8: 9.9 vs 8.4 us).
template <int BITS>
int choose_path(int M, int K, int64_t N) {
  int wk = 0, cpl = 0;
  if (BITS == 8 && sk8_shape(M, K) &&
      ((M >= 5 && M <= 8 && !(N <= 1024 && K >= 4096)) || (M <= 4 && M >= 3 && N >= 8192) ||
       (M >= 9 && !(K == 8192 && N > 16384))))
    return LOGBQ_PATH_SPLITK;
  if (sk_shape(M, K) && BITS == 4 &&
      ((M >= 5 && M <= 16) || (M == 4 && (N > 1024 || K <= 4096)) || (M == 3 && N >= 4096) ||
       (M > 16 && (K <= 4096 || N <= 16384 || M <= 20))))
    return LOGBQ_PATH_SPLITK;
  if (M <= 8 && gemv_config<BITS>(M, K, &wk, &cpl) &&
      !(M >= (BITS == 8 ? 5 : 3) && (int64_t)M * N > 65536))
    return LOGBQ_PATH_GEMV;
  if (BITS == 4 && kq_shape(M, N, K) && !narrow_fits(M, N)) return LOGBQ_PATH_MFMA_KQ;
  if (BITS == 8 && kq8_shape(M, N, K)) return LOGBQ_PATH_MFMA_KQ;
  return LOGBQ_PATH_MFMA;
}

// y_i = x . W_hat_i^T for up to kMaxSegs linears sharing x (validated by the caller).
template <int BITS>
int32_t run_linears(const uint16_t* x, int64_t m, int64_t k, const LinearJob* jobs, int count,
                    hipStream_t st) {
  int live[kMaxSegs];
  int nlive = 0;
  for (int i = 0; i < count; ++i)
    if (jobs[i].n > 0) live[nlive++] = i;
  if (m == 0 || nlive == 0) return LOGBQ_OK;
  const int cus = device_cus();
  if (cus <= 0) return LOGBQ_ERR_HIP;
  if (k == 0) {
    for (int a = 0; a < nlive; ++a) {
      const LinearJob& j = jobs[live[a]];
      fill_zero(j.y, m * j.n, cus, st);
      if (launch_status() != LOGBQ_OK) return LOGBQ_ERR_HIP;
    }
    return LOGBQ_OK;
  }
  const int M = (int)m, K = (int)k;
  int wk = 0, cpl = 0;
  int gl[kMaxSegs];
  int ng = 0;
  int64_t grows = 0;
  int sl[kMaxSegs];
  int ns = 0;
  for (int a = 0; a < nlive; ++a) {
    const LinearJob& j = jobs[live[a]];
    const int path = choose_path<BITS>(M, K, j.n);
    if (path == LOGBQ_PATH_SPLITK && BITS == 8) {
      const int32_t r = launch_sk8(x, M, K, j, st, cus);
      if (r != LOGBQ_OK) return r;
    } else if (path == LOGBQ_PATH_SPLITK) {
      sl[ns++] = live[a];
    } else if (path == LOGBQ_PATH_GEMV) {
      gl[ng++] = live[a];
      grows += j.n;
    } else if (path == LOGBQ_PATH_MFMA_KQ) {
      const int32_t r = BITS == 8 ? launch_kq8(x, M, K, j, st) : launch_kq(x, M, K, j, st);
      if (r != LOGBQ_OK) return r;
    } else {
      const int32_t r = launch_mfma<BITS>(x, M, K, j, st);
      if (r != LOGBQ_OK) return r;
    }
  }
  if (ns > 0) {
    const int32_t r = launch_sk(x, M, K, jobs, sl, ns, st, cus);
    if (r != LOGBQ_OK) return r;
  }
  if (ng == 0) return LOGBQ_OK;
  // The GEMV linears of the call share a launch when they take the same configuration (the
  // configuration depends only on (m, k, n), so each linear computes as in a call of its own).
  int cwk[kMaxSegs], ccpl[kMaxSegs];
  for (int a = 0; a < ng; ++a)
    if (!gemv_config_rows<BITS>(M, K, jobs[gl[a]].n, &cwk[a], &ccpl[a]))
      return LOGBQ_ERR_UNSUPPORTED;
  bool done[kMaxSegs] = {};
  for (int a0 = 0; a0 < ng; ++a0) {
    if (done[a0]) continue;
    wk = cwk[a0];
    cpl = ccpl[a0];
    int grp[kMaxSegs];
    int cnt = 0;
    grows = 0;
    for (int a = a0; a < ng; ++a)
      if (!done[a] && cwk[a] == wk && ccpl[a] == cpl) {
        grp[cnt++] = gl[a];
        grows += jobs[gl[a]].n;
        done[a] = true;
      }
    const int groups = 8 / wk;
    GemvSegs<BITS> segs;
    std::memset(&segs, 0, sizeof(segs));
    segs.count = cnt;
    int begin = 0;
    for (int a = 0; a < cnt; ++a) {
      const LinearJob& j = jobs[grp[a]];
      const int64_t need = (j.n + groups - 1) / groups;          // workgroups that have rows
      int64_t share = (int64_t)((double)cus * (double)j.n / (double)grows + 0.5);
      if (share < 1) share = 1;
      if (share > need) share = need;
      GemvSeg<BITS>& sg = segs.s[a];
      sg.codes = j.codes;
      sg.y = j.y;
      sg.n_rows = (int)j.n;
      sg.wg_begin = begin;
      const int64_t tg = share * groups;
      sg.iters = (int)((j.n + tg - 1) / tg);
      make_lut<BITS>(j.codebook, &sg.lut, &sg.scale);
      begin += (int)share;
    }
    const int stage_x = ((int64_t)M * K * 2 <= (int64_t)kStageXBytes) &&
                        !(M == 1 && cpl == 1 && wk == 1) ? 1 : 0;
    if (!dispatch_gemv<BITS>(M, cpl, begin, st, x, K, wk, stage_x, segs))
      return LOGBQ_ERR_UNSUPPORTED;
    if (launch_status() != LOGBQ_OK) return LOGBQ_ERR_HIP;
  }
  return LOGBQ_OK;
}

}  // namespace

// Error workspace of logbq_gptq_noalloc: [rows][128] float32 for at most kGptqScratchRows rows
// (8 MiB). It lives in the code object, so every device the library runs on holds its own copy
// until the process ends; host code reaches it only through the address hipGetSymbolAddress
// returns for the current device (the array's name is a host-side stand-in, not a device
// address).
constexpr int64_t kGptqScratchRows = 16384;
static __device__ __align__(256) float scratch[kGptqScratchRows * kGptqBlock];

// Device address of `scratch` on the current device, looked up once per device.
float* gptq_scratch_ptr() {
  static std::mutex mu;
  static void* ptrs[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (!ptrs[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    ptrs[dev] = p;
  }
  return static_cast<float*>(ptrs[dev]);
}

// One pass of the device fit: run the pass into its own region of the workspace (all regions
// are cleared by one fill before pass 1), copy its bins to the host and wait for them (the next
// pass's selection depends on them).
struct FitDeviceCtx {
  const float* w;
  int64_t n;
  unsigned long long* ws;
  hipStream_t st;
  std::vector<uint64_t> host;
};

// Workspace words: the pass-1 flags, then the bins of passes 1, 2 and 3.
constexpr int kFitOff1 = 1;
constexpr int kFitOff2 = kFitOff1 + 3 * logbq_detail::kFitBins1;
constexpr int kFitOff3 = kFitOff2 + 3 * logbq_detail::kFitBins2;
constexpr int kFitWords = kFitOff3 + 3 * logbq_detail::kFitBins3;
static_assert(kFitWords * 8 == LOGBQ_FIT_WORKSPACE_BYTES, "workspace size in the header");

int32_t fit_device_pass(void* vctx, int pass, uint32_t sel, logbq_detail::FitPassResult* res) {
  FitDeviceCtx& c = *static_cast<FitDeviceCtx*>(vctx);
  if (pass == 1) {
    hipLaunchKernelGGL(k_fill_u64, dim3((kFitWords + 255) / 256), dim3(256), 0, c.st, c.ws,
                       kFitWords);
    if (launch_status() != LOGBQ_OK) return LOGBQ_ERR_HIP;
  }
  const int cus = device_cus();
  if (cus <= 0) return LOGBQ_ERR_HIP;
  const int64_t chunk = fit_chunk(pass, c.n, cus);
  const unsigned grid = (unsigned)((c.n + chunk - 1) / chunk);
  unsigned int* flags = reinterpret_cast<unsigned int*>(c.ws);
  int off, words;
  if (pass == 1) {
    off = 0;   // the flags are copied with pass 1's bins
    words = kFitOff2;
    hipLaunchKernelGGL(k_fit_hist<1>, dim3(grid), dim3(kFitThreads), 0, c.st, c.w, c.n, chunk, sel,
                       c.ws + kFitOff1, flags);
  } else if (pass == 2) {
    off = kFitOff2;
    words = kFitOff3 - kFitOff2;
    hipLaunchKernelGGL(k_fit_hist<2>, dim3(grid), dim3(kFitThreads), 0, c.st, c.w, c.n, chunk, sel,
                       c.ws + kFitOff2, flags);
  } else {
    off = kFitOff3;
    words = kFitWords - kFitOff3;
    hipLaunchKernelGGL(k_fit_hist<3>, dim3(grid), dim3(kFitThreads), 0, c.st, c.w, c.n, chunk, sel,
                       c.ws + kFitOff3, flags);
  }
  if (launch_status() != LOGBQ_OK) return LOGBQ_ERR_HIP;
  c.host.assign((size_t)words, 0);
  if (hipMemcpyAsync(c.host.data(), c.ws + off, (size_t)words * 8, hipMemcpyDeviceToHost,
                     c.st) != hipSuccess)
    return LOGBQ_ERR_HIP;
  if (hipStreamSynchronize(c.st) != hipSuccess) return LOGBQ_ERR_HIP;
  if (pass == 1) {
    res->bins = c.host.data() + kFitOff1;
    res->max_key = (uint32_t)c.host[0];
    res->nonfinite = (uint32_t)(c.host[0] >> 32);
  } else {
    res->bins = c.host.data();
    res->max_key = 0;
    res->nonfinite = 0;
  }
  return LOGBQ_OK;
}

// Argument checks of the GPTQ entry points (everything but the device pointers) and the
// quantizer they describe.
int32_t gptq_validate(int64_t n, int64_t k, const logbq_params* p, const logbq_uniform* uniform,
                      GptqQuant* qz_out) {
  if (n < 0 || k < 0) return LOGBQ_ERR_INVALID_ARG;
  if ((p == nullptr) == (uniform == nullptr)) return LOGBQ_ERR_INVALID_ARG;
  if (k % 32 != 0) return LOGBQ_ERR_UNSUPPORTED;
  if (n > INT32_MAX || k > INT32_MAX || (n != 0 && (n * k) / n != k)) return LOGBQ_ERR_UNSUPPORTED;
  if (n > 65535LL * 16) return LOGBQ_ERR_UNSUPPORTED;   // rows are the after-block grid's y
  GptqQuant qz;
  std::memset(&qz, 0, sizeof(qz));
  if (p) {
    if (p->bits != 4 || p->qmax != 7) return LOGBQ_ERR_UNSUPPORTED;
    for (int i = 0; i < 16; ++i) qz.cb[i] = p->codebook[i];
    for (int i = 0; i < 7; ++i) qz.th[i] = p->thresholds[i];
    for (int i = 7; i < 15; ++i) qz.th[i] = INFINITY;
    qz.uniform = 0;
  } else {
    if (uniform->bits != 4) return LOGBQ_ERR_UNSUPPORTED;
    for (int i = 0; i < 16; ++i) qz.cb[i] = uniform->codebook[i];
    for (int i = 0; i < 15; ++i) qz.th[i] = uniform->thresholds[i];
    qz.uniform = 1;
  }
  for (int i = 0; i < 16; ++i)
    if (!std::isfinite(qz.cb[i])) return LOGBQ_ERR_INVALID_ARG;
  for (int i = 0; i < 15; ++i) {
    if (std::isnan(qz.th[i])) return LOGBQ_ERR_INVALID_ARG;
    if (i > 0 && qz.th[i] < qz.th[i - 1]) return LOGBQ_ERR_INVALID_ARG;
  }
  *qz_out = qz;
  return LOGBQ_OK;
}

// The column loop: per block of 128 columns, the panel kernel (quantize, in-block updates,
// errors into err_dev) and, unless it is the last block, the after-block kernel.
int32_t gptq_launch(float* w_dev, int N, int K, const float* u_dev, const GptqQuant& qz,
                    float* err_dev, uint8_t* codes_dev, hipStream_t st) {
  for (int i1 = 0; i1 < K; i1 += kGptqBlock) {
    const int nb = K - i1 < kGptqBlock ? K - i1 : kGptqBlock;
    hipLaunchKernelGGL(k_gptq_panel, dim3((unsigned)((N + 7) / 8)), dim3(512), 0, st, w_dev, N, K,
                       u_dev, i1, nb, qz, err_dev, codes_dev);
    if (launch_status() != LOGBQ_OK) return LOGBQ_ERR_HIP;
    if (i1 + nb < K) {
      hipLaunchKernelGGL(k_gptq_trail, dim3((unsigned)((K - i1 - nb + 63) / 64), (unsigned)((N + 15) / 16)),
                         dim3(256), 0, st, w_dev, N, K, u_dev, i1, nb, err_dev);
      if (launch_status() != LOGBQ_OK) return LOGBQ_ERR_HIP;
    }
  }
  return LOGBQ_OK;
}

extern "C" {

int32_t logbq_encode(const float* w_dev, int64_t n, int64_t k, const logbq_params* p,
                     uint8_t* codes_dev, float* codebook_out, void* stream) {
  if (!p || n < 0 || k < 0) return LOGBQ_ERR_INVALID_ARG;
  if (p->bits != 4 && p->bits != 8) return LOGBQ_ERR_UNSUPPORTED;
  if (k % 32 != 0) return LOGBQ_ERR_UNSUPPORTED;
  const int64_t numel = n * k;
  if (n != 0 && numel / n != k) return LOGBQ_ERR_UNSUPPORTED;
  if (numel > 0) {
    if (!w_dev || !codes_dev) return LOGBQ_ERR_INVALID_ARG;
    if (!aligned16(w_dev) || !aligned16(codes_dev)) return LOGBQ_ERR_UNSUPPORTED;
  }
  const int qmax = (1 << (p->bits - 1)) - 1;
  if (p->qmax != qmax) return LOGBQ_ERR_INVALID_ARG;
  for (int i = 0; i < qmax; ++i) {
    const float t = p->thresholds[i];
    if (std::isnan(t) || !(t > 0.0f)) return LOGBQ_ERR_INVALID_ARG;
    if (i > 0 && t < p->thresholds[i - 1]) return LOGBQ_ERR_INVALID_ARG;
  }
  if (codebook_out) std::memcpy(codebook_out, p->codebook, sizeof(float) << p->bits);
  if (numel == 0) return LOGBQ_OK;
  const int cus = device_cus();
  if (cus <= 0) return LOGBQ_ERR_HIP;
  const int64_t nchunk = numel / 4;
  // Workgroups per CU (the grid runs in several rounds): 64 (measured on the 8192x28672
  // tensor, 4-bit codes: 8 -> 190 us, 32 -> 183 us, 64 -> 178.5 us, 128 -> 181 us; 8-bit codes:
  // 32 -> 64 about 2 % faster).
  const int64_t grid = grid_for(nchunk, 256 * kEncU, (int64_t)cus * 64);
  if (p->bits == 4) {
    Thresholds th;
    for (int i = 0; i < 7; ++i) th.t[i] = p->thresholds[i];
    hipLaunchKernelGGL(k_encode, dim3((unsigned)grid), dim3(256), 0, (hipStream_t)stream,
                       reinterpret_cast<const f32x4*>(w_dev), reinterpret_cast<uint16_t*>(codes_dev),
                       nchunk, th);
  } else {
    Thresholds8 th;
    for (int i = 0; i < 127; ++i) th.t[i] = p->thresholds[i];
    th.inv = 0.0f;
    th.c = 0.0f;
    if (p->base > 1.0 && std::isfinite(p->base)) {
      // The device's float log2 and product add less than 0.1 step of error while
      // inv <= 1024 (b >= 2^(1/1024)) and |c| <= 2^20; with the quarter-step placement the
      // estimate is then never more than one step off.
      const double inv = 1.0 / std::log2(p->base), c = p->shift + 0.5;
      bool placed = inv <= 1024.0 && std::fabs(c) <= 1048576.0;
      for (int i = 0; i < 127 && placed; ++i) {
        const double f = std::log2((double)th.t[i]) * inv + c;
        placed = std::isfinite(f) && std::fabs(f - (i + 1)) < 0.25;
      }
      if (placed) {
        th.inv = (float)inv;
        th.c = (float)c;
      }
    }
    hipLaunchKernelGGL(k_encode8, dim3((unsigned)grid), dim3(256), 0, (hipStream_t)stream,
                       reinterpret_cast<const f32x4*>(w_dev), reinterpret_cast<uint32_t*>(codes_dev),
                       nchunk, th);
  }
  return launch_status();
}

int32_t logbq_encode_uniform(const float* w_dev, int64_t n, int64_t k, const logbq_uniform* u,
                             uint8_t* codes_dev, void* stream) {
  if (!u || n < 0 || k < 0) return LOGBQ_ERR_INVALID_ARG;
  if (u->bits != 4) return LOGBQ_ERR_UNSUPPORTED;
  if (k % 32 != 0) return LOGBQ_ERR_UNSUPPORTED;
  const int64_t numel = n * k;
  if (n != 0 && numel / n != k) return LOGBQ_ERR_UNSUPPORTED;
  for (int i = 0; i < 15; ++i) {
    const float t = u->thresholds[i];
    if (std::isnan(t)) return LOGBQ_ERR_INVALID_ARG;
    if (i > 0 && t < u->thresholds[i - 1]) return LOGBQ_ERR_INVALID_ARG;
  }
  if (numel == 0) return LOGBQ_OK;
  if (!w_dev || !codes_dev) return LOGBQ_ERR_INVALID_ARG;
  if (!aligned16(w_dev) || !aligned16(codes_dev)) return LOGBQ_ERR_UNSUPPORTED;
  const int cus = device_cus();
  if (cus <= 0) return LOGBQ_ERR_HIP;
  ThresholdsU th;
  for (int i = 0; i < 15; ++i) th.t[i] = u->thresholds[i];
  const int64_t nchunk = numel / 4;
  const int64_t grid = grid_for(nchunk, 256 * kEncU, (int64_t)cus * 64);
  hipLaunchKernelGGL(k_encode_uniform, dim3((unsigned)grid), dim3(256), 0, (hipStream_t)stream,
                     reinterpret_cast<const f32x4*>(w_dev), reinterpret_cast<uint16_t*>(codes_dev),
                     nchunk, th);
  return launch_status();
}

int32_t logbq_fit_device(const float* w_dev, int64_t numel, int32_t bits, double eps,
                         void* workspace_dev, logbq_params* out, void* stream) {
  if (!w_dev || !workspace_dev || !out || numel < 2) return LOGBQ_ERR_INVALID_ARG;
  if (!(eps > 0.0 && eps < 1.0)) return LOGBQ_ERR_INVALID_ARG;
  if (bits != 4 && bits != 8) return LOGBQ_ERR_UNSUPPORTED;
  if (numel >= (int64_t(1) << 40)) return LOGBQ_ERR_UNSUPPORTED;
  if (!aligned16(w_dev) || ((uintptr_t)workspace_dev & 7u) != 0) return LOGBQ_ERR_UNSUPPORTED;
  try {
    FitDeviceCtx c{w_dev, numel, static_cast<unsigned long long*>(workspace_dev),
                   (hipStream_t)stream, {}};
    return logbq_detail::fit_from_passes(bits, eps, fit_device_pass, &c, out);
  } catch (...) {   // host copies of the bins could not be allocated
    return LOGBQ_ERR_HOST_RESOURCE;
  }
}

int32_t logbq_gptq(float* w_dev, int64_t n, int64_t k, const float* u_dev, const logbq_params* p,
                   const logbq_uniform* uniform, float* err_dev, uint8_t* codes_dev,
                   void* stream) {
  GptqQuant qz;
  const int32_t v = gptq_validate(n, k, p, uniform, &qz);
  if (v != LOGBQ_OK || n == 0 || k == 0) return v;
  if (!w_dev || !u_dev || !err_dev || !codes_dev) return LOGBQ_ERR_INVALID_ARG;
  if (!aligned16(w_dev) || !aligned16(u_dev) || !aligned16(err_dev) || !aligned16(codes_dev))
    return LOGBQ_ERR_UNSUPPORTED;
  return gptq_launch(w_dev, (int)n, (int)k, u_dev, qz, err_dev, codes_dev, (hipStream_t)stream);
}

int32_t logbq_gptq_noalloc(float* w_dev, int64_t n, int64_t k, const float* u_dev,
                           const logbq_params* p, const logbq_uniform* uniform,
                           uint8_t* codes_dev, void* stream) {
  GptqQuant qz;
  const int32_t v = gptq_validate(n, k, p, uniform, &qz);
  if (v != LOGBQ_OK) return v;
  if (n > kGptqScratchRows) return LOGBQ_ERR_UNSUPPORTED;
  if (n == 0 || k == 0) return LOGBQ_OK;
  if (!w_dev || !u_dev || !codes_dev) return LOGBQ_ERR_INVALID_ARG;
  if (!aligned16(w_dev) || !aligned16(u_dev) || !aligned16(codes_dev))
    return LOGBQ_ERR_UNSUPPORTED;
  float* err = gptq_scratch_ptr();
  if (!err) return LOGBQ_ERR_HIP;
  return gptq_launch(w_dev, (int)n, (int)k, u_dev, qz, err, codes_dev, (hipStream_t)stream);
}

int32_t logbq_dequantize(const uint8_t* codes_dev, int64_t n, int64_t k, const float* codebook,
                         float* w_dev, void* stream) {
  if (!codebook || n < 0 || k < 0) return LOGBQ_ERR_INVALID_ARG;
  if (k % 32 != 0) return LOGBQ_ERR_UNSUPPORTED;
  const int64_t numel = n * k;
  if (n != 0 && numel / n != k) return LOGBQ_ERR_UNSUPPORTED;
  if (numel == 0) return LOGBQ_OK;
  if (!codes_dev || !w_dev) return LOGBQ_ERR_INVALID_ARG;
  if (!aligned16(codes_dev) || !aligned16(w_dev)) return LOGBQ_ERR_UNSUPPORTED;
  Codebook32 cb;
  std::memcpy(cb.v, codebook, sizeof(cb.v));
  const int cus = device_cus();
  if (cus <= 0) return LOGBQ_ERR_HIP;
  const int64_t nwords = numel / 8;
  const int64_t grid = grid_for(nwords, 256, (int64_t)cus * 16);
  hipLaunchKernelGGL(k_dequant, dim3((unsigned)grid), dim3(256), 0, (hipStream_t)stream,
                     reinterpret_cast<const uint32_t*>(codes_dev), reinterpret_cast<f32x4*>(w_dev),
                     nwords, cb);
  return launch_status();
}

int32_t logbq_linear(const uint16_t* x_dev, int64_t m, int64_t k, const uint8_t* codes_dev,
                     int64_t n, const float* codebook, float* y_dev, void* stream) {
  if (m < 0 || k < 0) return LOGBQ_ERR_INVALID_ARG;
  if (k % 32 != 0) return LOGBQ_ERR_UNSUPPORTED;
  if (m > kMaxBatchRows || k > INT32_MAX) return LOGBQ_ERR_UNSUPPORTED;
  LinearJob j{codes_dev, n, codebook, y_dev};
  const int32_t v = validate_job(j, m, k);
  if (v != LOGBQ_OK) return v;
  if (m == 0 || n == 0) return LOGBQ_OK;
  if (k > 0) {
    if (!x_dev) return LOGBQ_ERR_INVALID_ARG;
    if (!aligned16(x_dev)) return LOGBQ_ERR_UNSUPPORTED;
  }
  return run_linears<4>(x_dev, m, k, &j, 1, (hipStream_t)stream);
}

int32_t logbq_linear_multi(const uint16_t* x_dev, int64_t m, int64_t k, int32_t count,
                           const uint8_t* const* codes_dev, const int64_t* n,
                           const float* const* codebooks, float* const* y_dev, void* stream) {
  if (m < 0 || k < 0 || count < 1 || count > kMaxSegs) return LOGBQ_ERR_INVALID_ARG;
  if (!codes_dev || !n || !codebooks || !y_dev) return LOGBQ_ERR_INVALID_ARG;
  if (k % 32 != 0) return LOGBQ_ERR_UNSUPPORTED;
  if (m > kMaxBatchRows || k > INT32_MAX) return LOGBQ_ERR_UNSUPPORTED;
  LinearJob jobs[kMaxSegs];
  bool any = false;
  for (int i = 0; i < count; ++i) {
    jobs[i] = LinearJob{codes_dev[i], n[i], codebooks[i], y_dev[i]};
    const int32_t v = validate_job(jobs[i], m, k);
    if (v != LOGBQ_OK) return v;
    any = any || n[i] > 0;
  }
  if (m == 0 || !any) return LOGBQ_OK;
  if (k > 0) {
    if (!x_dev) return LOGBQ_ERR_INVALID_ARG;
    if (!aligned16(x_dev)) return LOGBQ_ERR_UNSUPPORTED;
  }
  return run_linears<4>(x_dev, m, k, jobs, count, (hipStream_t)stream);
}

int32_t logbq_linear8(const uint16_t* x_dev, int64_t m, int64_t k, const uint8_t* codes_dev,
                      int64_t n, const float* codebook, float* y_dev, void* stream) {
  if (m < 0 || k < 0) return LOGBQ_ERR_INVALID_ARG;
  if (k % 32 != 0) return LOGBQ_ERR_UNSUPPORTED;
  if (m > kMaxBatchRows || k > INT32_MAX) return LOGBQ_ERR_UNSUPPORTED;
  LinearJob j{codes_dev, n, codebook, y_dev};
  const int32_t v = validate_job(j, m, k, 256);
  if (v != LOGBQ_OK) return v;
  if (m == 0 || n == 0) return LOGBQ_OK;
  if (k > 0) {
    if (!x_dev) return LOGBQ_ERR_INVALID_ARG;
    if (!aligned16(x_dev)) return LOGBQ_ERR_UNSUPPORTED;
  }
  return run_linears<8>(x_dev, m, k, &j, 1, (hipStream_t)stream);
}

int32_t logbq_dequantize8(const uint8_t* codes_dev, int64_t n, int64_t k, const float* codebook,
                          float* w_dev, void* stream) {
  if (!codebook || n < 0 || k < 0) return LOGBQ_ERR_INVALID_ARG;
  if (k % 32 != 0) return LOGBQ_ERR_UNSUPPORTED;
  const int64_t numel = n * k;
  if (n != 0 && numel / n != k) return LOGBQ_ERR_UNSUPPORTED;
  if (numel == 0) return LOGBQ_OK;
  if (!codes_dev || !w_dev) return LOGBQ_ERR_INVALID_ARG;
  if (!aligned16(codes_dev) || !aligned16(w_dev)) return LOGBQ_ERR_UNSUPPORTED;
  const int cus = device_cus();
  if (cus <= 0) return LOGBQ_ERR_HIP;
  Codebook256 cb;
  std::memcpy(cb.v, codebook, sizeof(cb.v));
  const int64_t nwords = numel / 4;
  hipLaunchKernelGGL(k_dequant8, dim3((unsigned)grid_for(nwords, 256, (int64_t)cus * 16)),
                     dim3(256), 0, (hipStream_t)stream, reinterpret_cast<const uint32_t*>(codes_dev),
                     reinterpret_cast<f32x4*>(w_dev), nwords, cb);
  return launch_status();
}

int32_t logbq_linear_kernel(int32_t bits, int64_t m, int64_t k, int64_t n, const float* codebook,
                            char* name_out, int64_t name_len) {
  if (!name_out || name_len < 1 || m < 0 || k < 0 || n < 0) return LOGBQ_ERR_INVALID_ARG;
  if (bits != 4 && bits != 8) return LOGBQ_ERR_UNSUPPORTED;
  if (k % 32 != 0 || m > kMaxBatchRows || k > INT32_MAX || n > INT32_MAX)
    return LOGBQ_ERR_UNSUPPORTED;
  const int entries = 1 << bits;
  if (codebook)
    for (int i = 0; i < entries; ++i)
      if (!std::isfinite(codebook[i])) return LOGBQ_ERR_INVALID_ARG;
  char buf[96];
  if (m == 0 || n == 0) {
    std::snprintf(buf, sizeof(buf), "none");
  } else if (k == 0) {
    std::snprintf(buf, sizeof(buf), "k_fill_zero");
  } else {
    const int M = (int)m, K = (int)k;
    // Register dequantization needs a sign-symmetric codebook; every fitted one is, so a null
    // codebook stands for a fitted one.
    LutBytes tb;
    float scale;
    const bool symmetric = bits == 4 && (!codebook || make_lut_bytes(codebook, &tb, &scale));
    const int path = bits == 4 ? choose_path<4>(M, K, n) : choose_path<8>(M, K, n);
    int wk = 0, cpl = 0;
    if (path == LOGBQ_PATH_SPLITK && bits == 8) {
      std::snprintf(buf, sizeof(buf), "k_mfma_sk8<%d, %d>", K / 512, M <= 8 ? 2 : 1);
    } else if (path == LOGBQ_PATH_SPLITK && ((M <= 16 && K != 14336) || symmetric)) {
      const SkConfig c = sk_config(M, K, !symmetric, (int)((n + 15) / 16));
      std::snprintf(buf, sizeof(buf), "k_mfma_sk<%d, %d, %d, %d, %d, %s>", c.nd, c.waves,
                    c.groups, c.tiles, c.kparts, symmetric ? "false" : "true");
    } else if (path == LOGBQ_PATH_GEMV) {
      const bool ok = bits == 4 ? gemv_config_rows<4>(M, K, n, &wk, &cpl)
                                : gemv_config_rows<8>(M, K, n, &wk, &cpl);
      if (!ok) return LOGBQ_ERR_UNSUPPORTED;
      const int nbuf = (cpl <= 2 && M <= 2) ? 3 : 2;
      std::snprintf(buf, sizeof(buf), "k_gemv<%d, %d, %d, %s, %d>", bits, M, cpl,
                    wk > 1 ? "true" : "false", nbuf);
    } else if (path == LOGBQ_PATH_MFMA_KQ && bits == 8) {
      std::snprintf(buf, sizeof(buf), "k_mfma_kq8");
    } else if (path == LOGBQ_PATH_MFMA_KQ && symmetric) {
      std::snprintf(buf, sizeof(buf), "k_mfma_kq");
    } else {
      const StepCfg cfg = step_config(M, n, K, bits, symmetric);
      const int mt16 = cfg.mt16;
      if (cfg.narrow)
        std::snprintf(buf, sizeof(buf), "k_mfma2_narrow<%d, %d, %s, %s>", bits, mt16,
                      symmetric ? "false" : "true", mt16 <= 2 ? "true" : "false");
      else
        std::snprintf(buf, sizeof(buf), "k_mfma2<%d, %d, 4, %s, %s>", bits, mt16,
                      symmetric ? "false" : "true", mt16 <= 2 ? "true" : "false");
    }
  }
  const size_t need = std::strlen(buf) + 1;
  if ((int64_t)need > name_len) return LOGBQ_ERR_INVALID_ARG;
  std::memcpy(name_out, buf, need);
  return LOGBQ_OK;
}

int32_t logbq_linear_path(int32_t bits, int64_t m, int64_t k, int64_t n, int32_t* path_out) {
  if (!path_out || m < 0 || k < 0 || n < 0) return LOGBQ_ERR_INVALID_ARG;
  if (bits != 4 && bits != 8) return LOGBQ_ERR_UNSUPPORTED;
  if (k % 32 != 0 || m > kMaxBatchRows || k > INT32_MAX) return LOGBQ_ERR_UNSUPPORTED;
  if (m == 0 || n == 0 || k == 0) {
    *path_out = LOGBQ_PATH_NONE;
    return LOGBQ_OK;
  }
  *path_out = bits == 4 ? choose_path<4>((int)m, (int)k, n) : choose_path<8>((int)m, (int)k, n);
  return LOGBQ_OK;
}

}  // extern "C"
