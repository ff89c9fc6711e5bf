// GPU side of libsaki for gfx950 (CDNA4, wave64).
//
// Kernels (all on the caller's stream):
//   build_index_kernel   key codes c = B_k^T (k - mu) for every query head (Eq. 4)
//   score_batch_kernel   z = B_q^T q, b = q^T mu and s = z . c + b on MFMA for
//                        blocks of 16 query rows, top-64 per row (two passes:
//                        block maxima and a threshold, then the candidates)
//   score_scan_kernel    the same in one pass over the codes for long rows
//                        (batches of decode queries), running top-64 per row
//   score_stream_kernel  the same for few query rows per code set (decode):
//                        one key per lane, key range split into chunks
//   merge_kernel         reduces per-chunk partial top-64 lists of one row
//   keys_hi_kernel       bf16 hi/lo split of the keys and their norm bounds
//   exact_gate_kernel    exact top-64 and recall hits: float32 gate from the
//                        candidate list, bf16x3 MFMA scan, float64 decisions
//   exact_bf16_kernel, exact_mfma_kernel  fallback tiers of the same
//   exact_stream_kernel  exact float64 scores and top-64 for few query rows
//   moments_kernel       calibration moments in float64
//   attend_kernel        RoPE attention over the selected keys
//   export_kernel        debug read-back of the codes
// Top-k selection is in saki_topk.h.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <tuple>

#include <cfloat>
#include <climits>
#include <cmath>
#include <cstdint>
#include <type_traits>

#include "saki.h"
#include "saki_internal.h"
#include "saki_topk.h"

namespace {

using saki::kMaxK;
using saki::kTile;
using namespace saki_dev;

// MFMA operand and accumulator vectors
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef double f64x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) {
  bf16x8_t r;
  __builtin_memcpy(&r, &v, sizeof(r));
  return r;
}
__device__ __forceinline__ i16x4_t as_i16x4(uint2 v) {
  i16x4_t r;
  __builtin_memcpy(&r, &v, sizeof(r));
  return r;
}

constexpr int kStreamWaves = 4;  // waves per workgroup, streaming kernels
constexpr int kMfmaWaves = 2;    // waves per workgroup, MFMA kernels
constexpr int kMR = 16;          // query rows per wave on the MFMA kernels

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t bf16_bits(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}
__device__ __forceinline__ float bf16_round(float x) { return __uint_as_float(bf16_bits(x) << 16); }

// Storage types of the codes (template parameter ST of the index kernels).
constexpr int kStF32 = SAKI_F32, kStBf16 = SAKI_BF16, kStFp8 = SAKI_FP8;
template <int ST>
constexpr int code_bytes() { return ST == kStF32 ? 4 : ST == kStBf16 ? 2 : 1; }

// float32 -> fp8 E4M3 code: round to the nearest E4M3 value (ties to the even
// code), magnitudes of 448 and more saturate to 448 (finite inputs).
__device__ __forceinline__ uint32_t e4m3_bits(float x) {
  const uint32_t sign = (__float_as_uint(x) >> 24) & 0x80u;
  const float a = fabsf(x);
  if (!(a < 448.f)) return sign | 0x7Eu;
  if (a < 0x1p-6f) return sign | (uint32_t)rintf(a * 512.f);  // subnormal: multiples of 2^-9
  uint32_t u = __float_as_uint(a);
  u += 0x7FFFFu + ((u >> 20) & 1u);  // round the float32 significand to 3 bits, ties to even
  u &= 0xFFF00000u;
  const uint32_t code = (((u >> 23) - 120u) << 3) | ((u >> 20) & 7u);  // rebias 127 -> 7
  return sign | (code > 0x7Eu ? 0x7Eu : code);
}

// Four fp8 E4M3 codes (the bytes of w, lowest first) -> two words of bf16
// pairs.  Exact: an E4M3 value has at most 4 significant bits.
__device__ __forceinline__ uint2 e4m3x4_to_bf16(uint32_t w) {
  const auto lo = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, false);  // bytes 0, 1
  const auto hi = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, true);   // bytes 2, 3
  return uint2{(__float_as_uint(lo[0]) >> 16) | (__float_as_uint(lo[1]) & 0xffff0000u),
               (__float_as_uint(hi[0]) >> 16) | (__float_as_uint(hi[1]) & 0xffff0000u)};
}

template <bool BF>
__device__ __forceinline__ float load_key_elem(const void* p, size_t i) {
  if constexpr (BF) {
    const uint16_t v = reinterpret_cast<const uint16_t*>(p)[i];
    return __uint_as_float((uint32_t)v << 16);
  } else {
    return reinterpret_cast<const float*>(p)[i];
  }
}

// Key elements i .. i + 3 (i a multiple of 4) as floats.
template <bool BF>
__device__ __forceinline__ float4 load_key4(const void* p, size_t i) {
  if constexpr (BF) {
    const uint2 v = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(p) + i);
    return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                       __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u));
  } else {
    return *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(p) + i);
  }
}

// Unpack one 16-byte code piece into floats.
template <bool BF>
__device__ __forceinline__ void unpack_piece(uint4 v, float* out) {
  if constexpr (BF) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      out[2 * e] = __uint_as_float(w[e] << 16);
      out[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
    }
  } else {
    out[0] = __uint_as_float(v.x);
    out[1] = __uint_as_float(v.y);
    out[2] = __uint_as_float(v.z);
    out[3] = __uint_as_float(v.w);
  }
}

// Unpack one 16-byte piece of codes stored as ST into 16 / code_bytes<ST>() floats.
template <int ST>
__device__ __forceinline__ void unpack_codes(uint4 v, float* out) {
  if constexpr (ST == kStFp8) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint2 b = e4m3x4_to_bf16(w[e]);
      out[4 * e] = __uint_as_float(b.x << 16);
      out[4 * e + 1] = __uint_as_float(b.x & 0xffff0000u);
      out[4 * e + 2] = __uint_as_float(b.y << 16);
      out[4 * e + 3] = __uint_as_float(b.y & 0xffff0000u);
    }
  } else {
    unpack_piece<ST == kStBf16>(v, out);
  }
}

__device__ __forceinline__ int row_limit(int i, int Q, int N_valid, const int* q_pos) {
  if (i >= Q) return 0;
  if (!q_pos) return N_valid;
  const long long lim = (long long)q_pos[i] + 1;
  return lim < 0 ? 0 : (lim > N_valid ? N_valid : (int)lim);
}

// MI355X deals consecutive work-groups round-robin over its 8 XCDs, each with
// its own L2.  The MFMA kernels run on a 1-D grid of 8 * per_xcd work-groups
// and renumber them so that XCD x gets the contiguous logical range
// [x * per_xcd, (x + 1) * per_xcd): the row blocks of one head (which read the
// same codes / keys) then share one L2.  Returns -1 for padding work-groups.
constexpr int kXcds = 8;
__device__ __forceinline__ long long xcd_logical_block(long long total) {
  const long long hw = blockIdx.x;
  const long long per_xcd = (total + kXcds - 1) / kXcds;
  const long long logical = (hw % kXcds) * per_xcd + hw / kXcds;
  return logical < total ? logical : -1;
}

// Wave-wide max / min, returned in a scalar register (every lane holds the
// same value after the butterfly), so that what is derived from it stays on
// the scalar unit.
__device__ __forceinline__ int wave_max_i(int v) {
#pragma unroll
  for (int m = kWave / 2; m > 0; m >>= 1) v = max(v, __shfl_xor(v, m, kWave));
  return __builtin_amdgcn_readfirstlane(v);
}
__device__ __forceinline__ int wave_min_i(int v) {
#pragma unroll
  for (int m = kWave / 2; m > 0; m >>= 1) v = min(v, __shfl_xor(v, m, kWave));
  return __builtin_amdgcn_readfirstlane(v);
}

// max / min of floats as v_maximum3_f32 / v_minimum3_f32 (a NaN operand gives
// NaN; scores are never NaN), without the quieting moves fmaxf / fminf need.
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }
__device__ __forceinline__ float vmin(float a, float b) { return __builtin_elementwise_minimum(a, b); }

// Final list entry of a row -> output index / score.
template <class KO>
__device__ __forceinline__ int out_index(typename KO::K e) {
  const int j = KO::index(e);
  return j == kPadIdx ? -1 : j;
}

// Hits of an exact list (one entry per lane, the first k lanes count) against
// approx_idx row `row` (length k; entries < 0 never match).
__device__ __forceinline__ int row_hits(int ej, const int* __restrict__ approx, size_t row, int k) {
  const int lane = lane_id();
  const int aj = lane < k ? approx[row * k + lane] : -1;
  bool found = false;
  for (int m = 0; m < k; ++m) {
    const int v = __shfl(aj, m, kWave);
    found |= (v >= 0 && v == ej);
  }
  const bool counts = lane < k && ej >= 0 && found;
  return __popcll(__ballot(counts));
}

// ---------------------------------------------------------------- build index

// Key codes c_j = B_k^T (k_j - mu) on the bf16 MFMA (16x16x32).  Each float32
// operand is split into three bf16 terms: x = x1 + x2 + x3 with x1 = bf16(x),
// x2 = bf16(x - x1), x3 = bf16(x - x1 - x2) (each term takes the next 8
// significant bits, so the three carry a float32's 24), and likewise
// w = w1 + w2 + w3 for B_k.  The six products x_a w_b with a + b <= 4 are
// formed, x1 w1 into one float32 accumulator and the five smaller ones into a
// second; what is left out (x2 w3, x3 w2, x3 w3 and the splits' remainders)
// is below 4 * 2^-24 |x| |w| per element, the size of float32 rounding, at
// 6 bf16 products where float32 operands would take 16 times the MFMA time of
// one.  A work-group takes a slice of the keys of one KV head (16-key groups,
// taken by its 8 waves in turn) and computes their codes for every query head of the group, so
// each key is read once (a short range, a decode append, takes one query head
// per work-group instead, so that the heads' factors load in parallel).  For
// a group of 16 keys and a block of 16 code dimensions the MFMA forms
// D[m][key] = sum_c B_k[c][m] (k - mu)[key][c] in 4 steps of 32 dimensions:
// lane (key qi, group g) loads dims 32 kk + 8 g .. + 7 of its key (the B
// operand) and of B_k's column m = 16 mc + qi (the A operand).  The three
// terms of B_k of up to build_heads_lds<r>() heads at a time sit in LDS,
// transposed (one row of 128 dims per code dimension, rows of 136 bf16 so
// that the 16 rows one read touches start 4 banks apart).  Lane (qi, g) ends
// with dims 16 mc + 4 g .. + 3 of key qi: one 16-byte float32 piece, half a
// bf16 piece or a quarter of an fp8 piece.  Centring is float32 (k - mu)
// before the product, as the paper writes it.
constexpr int kBuildKeys = 1024;         // keys per work-group, at least
constexpr int kBuildSplitKeys = 256;     // ranges up to this many keys: one query head per work-group
constexpr int kBuildRounds = 1;          // work-groups per slot the device holds
constexpr int kBuildRow = 136;           // bf16 per LDS row of B_k (128 dims + 8)
constexpr int kBuildLdsBytes = 104448;   // B_k of up to 4 heads at r = 32
template <int RK>
constexpr int build_heads_lds() { return kBuildLdsBytes / (3 * RK * kBuildRow * 2); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two floats rounded to bf16 (nearest even, v_cvt_pk_bf16_f32), packed low
// first.
__device__ __forceinline__ uint32_t bf16x2_bits(float a, float b) {
  const bf16x2_t v = __builtin_convertvector(f32x2_t{a, b}, bf16x2_t);
  uint32_t u;
  __builtin_memcpy(&u, &v, sizeof(u));
  return u;
}

// Splits a pair of floats into three packed bf16 pairs t[0] + t[1] + t[2].
__device__ __forceinline__ void split3_bf16x2(float a, float b, uint32_t t[3]) {
#pragma unroll
  for (int p = 0; p < 3; ++p) {
    t[p] = bf16x2_bits(a, b);
    a -= __uint_as_float(t[p] << 16);
    b -= __uint_as_float(t[p] & 0xffff0000u);
  }
}

// grid (slices, H_kv or H_q (per_head), B), block 64 * kBuildWaves; the keys
// [n_begin rounded down to 16, n_end) are cut into gridDim.x contiguous
// slices, one per work-group, so that B_k is staged in LDS once per slice.
constexpr int kBuildWaves = 8;
template <int RK, bool KBF, int ST>
__global__ __launch_bounds__(kBuildWaves * kWave) void build_index_kernel(
    const void* __restrict__ keys, const float* __restrict__ Bk,
    const float* __restrict__ mu, int H_q, int H_kv, int N_cap, int n_tiles,
    uint8_t* __restrict__ index, int n_begin, int n_end, int per_head) {
  constexpr int D = saki::kHeadDim;
  constexpr int ES = code_bytes<ST>();
  constexpr int HB = build_heads_lds<RK>();
  static_assert(HB >= 1, "one head of B_k fits");
  constexpr size_t TB = (size_t)kTile * RK * ES;  // bytes of one 64-key tile
  constexpr int NM = RK / 16;
  constexpr int SG = 2;                // 16-key groups per wave step
  constexpr int MB = NM < 2 ? NM : 2;  // 16-dim code blocks per pass over a step's keys
  constexpr int PS = RK * kBuildRow;  // bf16 per term of one head
  __shared__ __align__(16) uint16_t bks[HB * 3 * PS];
  const int G = H_q / H_kv;
  const int gkv = per_head ? (int)blockIdx.y / G : (int)blockIdx.y, b = blockIdx.z;
  const int h_first = per_head ? (int)blockIdx.y : gkv * G;  // query heads [h_first, h_end)
  const int h_end = per_head ? h_first + 1 : h_first + G;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int qi = lane % 16, g = lane / 16;
  // this work-group's keys [k0, k1): slices of the range from n_begin rounded
  // down to 16, a multiple of 16 keys each
  const int kb = (n_begin / 16) * 16;
  const int slice = ((n_end - kb + (int)gridDim.x - 1) / (int)gridDim.x + 15) / 16 * 16;
  const int k0 = kb + (int)blockIdx.x * slice;
  if (k0 >= n_end) return;  // the whole work-group
  const int k1 = min(n_end, k0 + slice);
  const size_t key_base = ((size_t)b * H_kv + gkv) * N_cap;
  __shared__ __align__(16) float mus[D];  // mu of the KV head (read after the first barrier below)
  if (tid < D / 4)
    reinterpret_cast<float4*>(mus)[tid] = reinterpret_cast<const float4*>(mu + (size_t)gkv * D)[tid];
  // raw key dims 32 kk + 8 g .. + 7 of key n (16 bytes of bf16 or 32 of float32 per kk)
  struct RawKey {
    uint4 v[KBF ? 4 : 8];
  };
  auto load_raw = [&](int n, bool ok, RawKey& r) {
#pragma unroll
    for (int i = 0; i < (KBF ? 4 : 8); ++i) {
      const size_t off = (key_base + n) * D + (KBF ? 32 * i + 8 * g : 32 * (i / 2) + 8 * g + 4 * (i % 2));
      r.v[i] = ok ? (KBF ? *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(keys) + off)
                         : *reinterpret_cast<const uint4*>(reinterpret_cast<const float*>(keys) + off))
                  : uint4{0u, 0u, 0u, 0u};
    }
  };
  // (k - mu) split into three bf16 terms: xp[p][kk] holds dims 32 kk + 8 g .. + 7
  auto split_key = [&](const RawKey& r, bool ok, uint4 xp[3][4]) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      float f[8];
      if constexpr (KBF) {
        unpack_piece<true>(r.v[kk], f);
      } else {
        unpack_piece<false>(r.v[2 * kk], f);
        unpack_piece<false>(r.v[2 * kk + 1], f + 4);
      }
      float m[8];
      *reinterpret_cast<float4*>(m) = *reinterpret_cast<const float4*>(&mus[32 * kk + 8 * g]);
      *reinterpret_cast<float4*>(m + 4) = *reinterpret_cast<const float4*>(&mus[32 * kk + 8 * g + 4]);
      uint32_t t[4][3];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        split3_bf16x2(ok ? f[2 * e] - m[2 * e] : 0.f, ok ? f[2 * e + 1] - m[2 * e + 1] : 0.f, t[e]);
#pragma unroll
      for (int p = 0; p < 3; ++p) xp[p][kk] = uint4{t[0][p], t[1][p], t[2][p], t[3][p]};
    }
  };
  // code dims 16 (mc0 + mc) + 4 g .. + 3 of key n, mc < MB
  auto store = [&](int n, int h, int mc0, const f32x4_t* acc) {
    uint8_t* tb = index + (((size_t)b * H_q + h) * n_tiles + n / kTile) * TB;
#pragma unroll
    for (int mc = 0; mc < MB; ++mc) {
      const int m = 16 * (mc0 + mc) + 4 * g;  // first code dim of this lane
      uint8_t* dst = tb + (size_t)(m * ES / 16) * kTile * 16 + (size_t)(n % kTile) * 16 + (m * ES) % 16;
      const f32x4_t v = acc[mc];
      if constexpr (ST == kStFp8) {
        *reinterpret_cast<uint32_t*>(dst) = e4m3_bits(v[0]) | (e4m3_bits(v[1]) << 8) |
                                            (e4m3_bits(v[2]) << 16) | (e4m3_bits(v[3]) << 24);
      } else if constexpr (ST == kStBf16) {
        *reinterpret_cast<uint2*>(dst) =
            uint2{bf16_bits(v[0]) | (bf16_bits(v[1]) << 16), bf16_bits(v[2]) | (bf16_bits(v[3]) << 16)};
      } else {
        *reinterpret_cast<uint4*>(dst) = uint4{__float_as_uint(v[0]), __float_as_uint(v[1]),
                                               __float_as_uint(v[2]), __float_as_uint(v[3])};
      }
    }
  };
  // a wave takes SG groups of 16 keys per step, so that each B_k operand read
  // from LDS serves SG products
  const int n_steps = (k1 - k0 + 16 * SG - 1) / (16 * SG);
  auto key_at = [&](int st, int sg) { return k0 + 16 * (SG * st + sg) + qi; };
  auto key_ok = [&](int n) { return n >= n_begin && n < k1; };
  constexpr int NT = kBuildWaves * kWave;
  constexpr int FB = 4;  // B_k pairs per thread whose loads are issued together
  for (int h0 = h_first; h0 < h_end; h0 += HB) {
    const int nh = min(HB, h_end - h0);
    __syncthreads();  // the previous heads' reads are done
    // B_k[h][c][m] (row-major D x RK) -> term p at bks[((hh * 3 + p) * RK + m) * kBuildRow + c],
    // dims c = 2 c2, 2 c2 + 1 per pair
    for (int e0 = tid; e0 < nh * (D / 2) * RK; e0 += FB * NT) {
      float2 w[FB];
#pragma unroll
      for (int i = 0; i < FB; ++i) {
        const int e = e0 + i * NT;
        const int m = e % RK, c2 = (e / RK) % (D / 2), hh = e / (RK * (D / 2));
        const float* src = Bk + ((size_t)(h0 + hh) * D + 2 * c2) * RK + m;
        w[i] = e < nh * (D / 2) * RK ? make_float2(src[0], src[RK]) : make_float2(0.f, 0.f);
      }
#pragma unroll
      for (int i = 0; i < FB; ++i) {
        const int e = e0 + i * NT;
        const int m = e % RK, c2 = (e / RK) % (D / 2), hh = e / (RK * (D / 2));
        uint32_t t[3];
        split3_bf16x2(w[i].x, w[i].y, t);
        if (e < nh * (D / 2) * RK)
#pragma unroll
          for (int p = 0; p < 3; ++p)
            *reinterpret_cast<uint32_t*>(&bks[((hh * 3 + p) * RK + m) * kBuildRow + 2 * c2]) = t[p];
      }
    }
    __syncthreads();
    RawKey cur[SG];
    if (wave < n_steps)
#pragma unroll
      for (int sg = 0; sg < SG; ++sg) load_raw(key_at(wave, sg), key_ok(key_at(wave, sg)), cur[sg]);
    for (int st = wave; st < n_steps; st += kBuildWaves) {
      uint4 xp[SG][3][4];
#pragma unroll
      for (int sg = 0; sg < SG; ++sg) split_key(cur[sg], key_ok(key_at(st, sg)), xp[sg]);
      if (st + kBuildWaves < n_steps)  // the wave's next step, loaded under this one's products
#pragma unroll
        for (int sg = 0; sg < SG; ++sg)
          load_raw(key_at(st + kBuildWaves, sg), key_ok(key_at(st + kBuildWaves, sg)), cur[sg]);
#pragma unroll 1
      for (int hm = 0; hm < nh * (NM / MB); ++hm) {  // head hh, code dims from 16 mc0
        const int hh = hm / (NM / MB), mc0 = (hm % (NM / MB)) * MB;
        f32x4_t hi[SG][MB], lo[SG][MB];
#pragma unroll
        for (int sg = 0; sg < SG; ++sg)
#pragma unroll
          for (int mc = 0; mc < MB; ++mc) {
            hi[sg][mc] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            lo[sg][mc] = f32x4_t{0.f, 0.f, 0.f, 0.f};
          }
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          // the operands of one 32-dim step at a time (register room)
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int mc = 0; mc < MB; ++mc) {
            const uint16_t* wr = &bks[(hh * 3 * RK + 16 * (mc0 + mc) + qi) * kBuildRow + 32 * kk + 8 * g];
            const bf16x8_t w1 = as_bf16x8(*reinterpret_cast<const uint4*>(wr));
            const bf16x8_t w2 = as_bf16x8(*reinterpret_cast<const uint4*>(wr + PS));
            const bf16x8_t w3 = as_bf16x8(*reinterpret_cast<const uint4*>(wr + 2 * PS));
#pragma unroll
            for (int sg = 0; sg < SG; ++sg) {
              const bf16x8_t x1 = as_bf16x8(xp[sg][0][kk]), x2 = as_bf16x8(xp[sg][1][kk]),
                             x3 = as_bf16x8(xp[sg][2][kk]);
              hi[sg][mc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w1, x1, hi[sg][mc], 0, 0, 0);
              lo[sg][mc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w3, x1, lo[sg][mc], 0, 0, 0);
              lo[sg][mc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w2, x2, lo[sg][mc], 0, 0, 0);
              lo[sg][mc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w1, x3, lo[sg][mc], 0, 0, 0);
              lo[sg][mc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w2, x1, lo[sg][mc], 0, 0, 0);
              lo[sg][mc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w1, x2, lo[sg][mc], 0, 0, 0);
            }
          }
        }
#pragma unroll
        for (int sg = 0; sg < SG; ++sg) {
#pragma unroll
          for (int mc = 0; mc < MB; ++mc) hi[sg][mc] += lo[sg][mc];
          const int n = key_at(st, sg);
          if (key_ok(n)) store(n, h0 + hh, mc0, hi[sg]);
        }
      }
    }
  }
}

// grid (tiles, B*H_q), block 64: codes -> float [B, H_q, N_cap, r].
template <int RK, int ST>
__global__ __launch_bounds__(64) void export_kernel(const uint8_t* __restrict__ index,
                                                    int n_tiles, int N_cap,
                                                    float* __restrict__ out) {
  constexpr int ES = code_bytes<ST>();
  constexpr int CPP = saki::kChunkBytes / ES;
  constexpr int NP = RK / CPP;
  const int tile = blockIdx.x;
  const size_t bh = blockIdx.y;
  const int t = threadIdx.x;
  const int n = tile * kTile + t;
  if (n >= N_cap) return;
  const uint8_t* tbase = index + (bh * n_tiles + tile) * ((size_t)kTile * RK * ES);
  for (int piece = 0; piece < NP; ++piece) {
    const uint4 v = *reinterpret_cast<const uint4*>(tbase + (size_t)piece * kTile * 16 + (size_t)t * 16);
    float f[CPP];
    unpack_codes<ST>(v, f);
    for (int e = 0; e < CPP; ++e) out[(bh * N_cap + n) * RK + piece * CPP + e] = f[e];
  }
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ bf16x2_t as_bf16x2(uint32_t v) {
  bf16x2_t r;
  __builtin_memcpy(&r, &v, sizeof(r));
  return r;
}

// ---------------------------------------------------------------- sketch scoring, streaming

// grid (row_blocks * n_chunks, B * index_heads), block 64*waves.  The rows of
// a code set are its gq = H_q / index_heads query heads times the Q queries,
// numbered rho = i * gq + (h % gq) so that one wave's R rows are the heads
// sharing the codes (for a GQA-shared index) before further queries.  Each
// wave owns R rows and one key chunk; lane t scores key t of each 64-key tile.
// With `split` (fewer than four waves' worth of rows per code set) the four
// waves of a work-group share their R rows and take four consecutive chunks.
// The query sketch of the rows (Sec. 6: z = B_q^T q, rounded to bf16 for bf16
// and fp8 codes, and b = q^T mu, float32 sums) is formed before the scan: by
// the four waves together when they share rows (wave w sums dims 32w ..
// 32w + 31, the four partial sums are added in wave order), otherwise by
// each wave for its own rows (dims in order).  The first code tiles are
// requested before the sketch, so that its loads wait under theirs.
template <int RK, int ST, int R>
__global__ __launch_bounds__(256) void score_stream_kernel(
    const uint8_t* __restrict__ index, int n_tiles, int N_valid, int Q,
    const int* __restrict__ q_pos, const float* __restrict__ q, const float* __restrict__ Bq,
    const float* __restrict__ mu, int H_q, int H_kv, int gq, int row_blocks, int chunk,
    int n_chunks, int split, int k, int* __restrict__ top_idx, float* __restrict__ top_score,
    uint64_t* __restrict__ part) {
  constexpr int ES = code_bytes<ST>();
  constexpr int CPP = saki::kChunkBytes / ES;
  constexpr int NP = RK / CPP;
  constexpr size_t TB = (size_t)kTile * RK * ES;
  using KO = KeysF32;
  constexpr int D = saki::kHeadDim;
  constexpr int NO = R * (RK + 1);  // sketch outputs of R rows
  __shared__ float zs[kStreamWaves][R][RK + 1];  // element RK: the mean term b
  __shared__ float zpart[kStreamWaves][NO];      // split: partial sums of wave w
  __shared__ uint64_t lmem[kStreamWaves][R][kList];
  __shared__ uint64_t bmem[kStreamWaves][R][kList];
  // the wave index is uniform over the wave: say so, so that what depends on
  // it (the sketch's dim slice, the chunk) stays in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = lane_id();
  const int waves = blockDim.x / kWave;
  const int rb = blockIdx.x % row_blocks;
  const int ch = split ? (blockIdx.x / row_blocks) * waves + wave : blockIdx.x / row_blocks;
  const size_t bi = blockIdx.y;  // b * index_heads + code set
  const int index_heads = H_q / gq;
  const size_t b = bi / index_heads;
  const int ih = (int)(bi % index_heads);
  const int n_rho = gq * Q;
  const int row0 = split ? rb * R : (rb * waves + wave) * R;
  if (row0 >= n_rho) return;  // never with split (row_blocks = ceil(n_rho / R))

  int lim[R];
  size_t flat[R];  // (b * H_q + h) * Q + i of each row
  int kmax = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int rho = row0 + r;
    const bool ok = rho < n_rho;
    const int i = ok ? rho / gq : 0;
    const int h = ih * gq + (ok ? rho % gq : 0);
    flat[r] = (b * H_q + h) * Q + i;
    lim[r] = ok ? row_limit(i, Q, N_valid, q_pos) : 0;
    kmax = lim[r] > kmax ? lim[r] : kmax;
  }
  RowLists<KO, R> top;
  top.init(&lmem[wave][0][0], &bmem[wave][0][0]);

  const int kbeg = ch * chunk;
  const int kend = min(kbeg + chunk, kmax);
  const uint8_t* hbase = index + bi * n_tiles * TB;
  // the next tile's pieces are loaded before this tile is scored (sketches of
  // up to 128 bytes per key; wider ones are loaded as they are used)
  constexpr int PF = NP <= 8 ? NP : 1;
  uint4 nxt[PF];
  auto load_tile = [&](int t0, uint4* v) {
    const uint8_t* tb = hbase + (size_t)(t0 / kTile) * TB + (size_t)lane * 16;
#pragma unroll
    for (int p = 0; p < PF; ++p) v[p] = *reinterpret_cast<const uint4*>(tb + (size_t)p * kTile * 16);
  };
  // with at most 32 bytes of bf16 or fp8 code per key, two tiles are loaded
  // ahead (into two buffers taken in turn) so that as many bytes are in
  // flight as for wider codes; otherwise one
  constexpr int kAhead = ST != kStF32 && NP * 16 <= 32 ? 2 : 1;
  uint4 nxt2[PF];
  if (kbeg < kend) load_tile(kbeg, nxt);
  if (kAhead == 2 && kbeg + kTile < kend) load_tile(kbeg + kTile, nxt2);
  // the query sketch: output o = r * (RK + 1) + m of the rows in lane o % 64
  // (m < RK: z_m, m = RK: b), loads taken 16 dims at a time
  if (split) {
    constexpr int DS = D / kStreamWaves;
    static_assert(DS % 16 == 0, "dim slices of whole load groups");
    for (int o0 = 0; o0 < NO; o0 += kWave) {
      const int o = o0 + lane;
      const int r = R == 1 ? 0 : min(o / (RK + 1), R - 1), m = o % (RK + 1);
      const int rho = row0 + r;
      const bool rv = rho < n_rho;
      const int i = rv ? rho / gq : 0;
      const int h = ih * gq + (rv ? rho % gq : 0);
      const int stride = m < RK ? RK : 1;
      const float* qv = q + ((b * H_q + h) * Q + i) * D + wave * DS;
      const float* col = (m < RK ? Bq + (size_t)h * D * RK + m : mu + (size_t)(h / (H_q / H_kv)) * D) +
                         (size_t)wave * DS * stride;
      float acc = 0.f;
#pragma unroll 1
      for (int c0 = 0; c0 < DS; c0 += 16) {
        float qa[16], ba[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          qa[u] = qv[c0 + u];
          ba[u] = col[(size_t)(c0 + u) * stride];
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) acc = fmaf(qa[u], ba[u], acc);
      }
      if (o < NO) zpart[wave][o] = acc;
    }
    __syncthreads();
    for (int o = lane; o < NO; o += kWave) {
      const int r = o / (RK + 1), m = o % (RK + 1);
      float v = ((zpart[0][o] + zpart[1][o]) + zpart[2][o]) + zpart[3][o];
      if (ST != kStF32 && m < RK) v = bf16_round(v);
      zs[wave][r][m] = row0 + r < n_rho ? v : 0.f;
    }
    wave_lds_sync();
  } else {
    constexpr int CG = 16;
    for (int o0 = 0; o0 < NO; o0 += kWave) {
      const int o = o0 + lane;
      // with one row per wave the query row is the same in every lane
      const int r = R == 1 ? 0 : min(o / (RK + 1), R - 1), m = o % (RK + 1);
      const int rho = row0 + r;
      const bool rv = rho < n_rho;
      const bool ok = o < NO && rv;
      const int i = rv ? rho / gq : 0;
      const int h = ih * gq + (rv ? rho % gq : 0);
      const float* qv = q + ((b * H_q + h) * Q + i) * D;
      const float* col = m < RK ? Bq + (size_t)h * D * RK + m : mu + (size_t)(h / (H_q / H_kv)) * D;
      const int stride = m < RK ? RK : 1;
      float acc = 0.f;
#pragma unroll 1
      for (int c0 = 0; c0 < D; c0 += CG) {
        float qa[CG], ba[CG];
#pragma unroll
        for (int u = 0; u < CG; ++u) {
          qa[u] = qv[c0 + u];
          ba[u] = col[(size_t)(c0 + u) * stride];
        }
#pragma unroll
        for (int u = 0; u < CG; ++u) acc = fmaf(qa[u], ba[u], acc);
      }
      if (ST != kStF32 && m < RK) acc = bf16_round(acc);
      if (o < NO) zs[wave][r][m] = ok ? acc : 0.f;
    }
    wave_lds_sync();
  }
  float bb[R];
#pragma unroll
  for (int r = 0; r < R; ++r) bb[r] = zs[wave][r][RK];
  if constexpr (ST != kStF32) {
    // bf16 codes: each 32-bit word holds elements (2e, 2e + 1), scored with
    // the packed bf16 dot product against the query sketch's pairs; fp8
    // codes are first widened to such words (exactly)
    // the pairs are the same in every lane: when they fit, scalar registers
    // hold them and the vector registers are left to the key tiles
    constexpr bool kScalarZ = R * RK / 2 <= 64;
    uint32_t zp[R][RK / 2];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int m = 0; m < RK / 2; ++m) {
        const uint32_t v = (__float_as_uint(zs[wave][r][2 * m]) >> 16) |
                           (__float_as_uint(zs[wave][r][2 * m + 1]) & 0xffff0000u);
        zp[r][m] = kScalarZ ? (uint32_t)__builtin_amdgcn_readfirstlane((int)v) : v;
      }
    // one tile: the words of bf16 pairs from `cur` (and the pieces not
    // prefetched), then `refill` (which may reload cur's registers), then the
    // dot products
    auto tile = [&](int t0, const uint4* cur, auto&& refill) {
      const int j = t0 + lane;
      const uint8_t* tb = hbase + (size_t)(t0 / kTile) * TB;
      uint32_t w[RK / 2];
      auto put = [&](int p, const uint4& v) {  // piece p -> its words of bf16 pairs
        if constexpr (ST == kStFp8) {
          const uint32_t vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint2 bw = e4m3x4_to_bf16(vv[e]);
            w[8 * p + 2 * e] = bw.x;
            w[8 * p + 2 * e + 1] = bw.y;
          }
        } else {
          w[4 * p] = v.x; w[4 * p + 1] = v.y; w[4 * p + 2] = v.z; w[4 * p + 3] = v.w;
        }
      };
#pragma unroll
      for (int p = 0; p < PF; ++p) put(p, cur[p]);
#pragma unroll
      for (int p = PF; p < NP; ++p)
        put(p, *reinterpret_cast<const uint4*>(tb + (size_t)p * kTile * 16 + (size_t)lane * 16));
      refill();
#pragma unroll
      for (int r = 0; r < R; ++r) {
        float acc = 0.f;
#pragma unroll
        for (int m = 0; m < RK / 2; ++m) acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(w[m]), as_bf16x2(zp[r][m]), acc, false);
        top.offer(r, j < lim[r] ? acc + bb[r] : -INFINITY, j);
      }
    };
    if constexpr (kAhead == 2) {
      for (int t0 = kbeg; t0 < kend; t0 += 2 * kTile) {
        tile(t0, nxt, [&] { if (t0 + 2 * kTile < kend) load_tile(t0 + 2 * kTile, nxt); });
        if (t0 + kTile >= kend) break;
        tile(t0 + kTile, nxt2, [&] { if (t0 + 3 * kTile < kend) load_tile(t0 + 3 * kTile, nxt2); });
      }
    } else {
      for (int t0 = kbeg; t0 < kend; t0 += kTile)
        tile(t0, nxt, [&] { if (t0 + kTile < kend) load_tile(t0 + kTile, nxt); });
    }
  } else {
    for (int t0 = kbeg; t0 < kend; t0 += kTile) {
      const int j = t0 + lane;
      const uint8_t* tb = hbase + (size_t)(t0 / kTile) * TB;
      float c[RK];
#pragma unroll
      for (int p = 0; p < PF; ++p) unpack_codes<ST>(nxt[p], c + p * CPP);
#pragma unroll
      for (int p = PF; p < NP; ++p) {
        const uint4 v = *reinterpret_cast<const uint4*>(tb + (size_t)p * kTile * 16 + (size_t)lane * 16);
        unpack_codes<ST>(v, c + p * CPP);
      }
      if (t0 + kTile < kend) load_tile(t0 + kTile, nxt);
#pragma unroll
      for (int r = 0; r < R; ++r) {
        float acc = 0.f;
#pragma unroll
        for (int m = 0; m < RK; ++m) acc = fmaf(zs[wave][r][m], c[m], acc);
        top.offer(r, j < lim[r] ? acc + bb[r] : -INFINITY, j);
      }
    }
  }
  for (int r = 0; r < R; ++r) {
    top.finish(r);
    if (row0 + r >= n_rho || ch >= n_chunks) continue;  // a split wave past the last chunk
    const uint64_t e = top.entry(r);
    if (n_chunks == 1) {
      if (lane < k) {
        const size_t o = flat[r] * k + lane;
        top_idx[o] = out_index<KO>(e);
        if (top_score) top_score[o] = KO::score(e);
      }
    } else {
      part[(flat[r] * n_chunks + ch) * kMaxK + lane] = e;
    }
  }
}

// ---------------------------------------------------------------- sketch scoring, MFMA

// Query blocks of 16 rows per wave, the column count of the 16x16 MFMA tiles.
// A = 16 keys of the current tile (rows), B = the wave's 16 queries (columns),
// so each lane holds scores of one query (lane % 16) against 16 keys of every
// 64-key tile.  The scorer and the query-sketch prologue below serve the
// batched kernel (score_batch_kernel), the one-pass kernel for long rows
// (score_scan_kernel) and the exact-recall kernels.

// Pack 8 floats that already hold bf16 values into a bf16x8 operand.
__device__ __forceinline__ uint4 pack_bf16x8(const float* f) {
  uint4 u;
  u.x = (__float_as_uint(f[0]) >> 16) | (__float_as_uint(f[1]) & 0xffff0000u);
  u.y = (__float_as_uint(f[2]) >> 16) | (__float_as_uint(f[3]) & 0xffff0000u);
  u.z = (__float_as_uint(f[4]) >> 16) | (__float_as_uint(f[5]) & 0xffff0000u);
  u.w = (__float_as_uint(f[6]) >> 16) | (__float_as_uint(f[7]) & 0xffff0000u);
  return u;
}
__device__ __forceinline__ float xor_shfl_f32(float v, int m) {
  return __uint_as_float(xor_shfl_u32(__float_as_uint(v), m));
}
// Sum over the four lanes that share lane % 16.
__device__ __forceinline__ float sum_lane_groups(float v) {
  v += xor_shfl_f32(v, 16);
  return v + xor_shfl_f32(v, 32);
}

// Upper-tail standard normal quantile: z with P(X > z) = tail, tail in (0, 0.5]
// (Abramowitz & Stegun 26.2.23, absolute error below 4.5e-4).  Only used to
// predict where a row's 64th score lies.
__device__ __forceinline__ float normal_upper_quantile(float tail) {
  const float t = sqrtf(-2.f * __logf(tail));
  return t - (2.515517f + t * (0.802853f + t * 0.010328f)) /
                 (1.f + t * (1.432788f + t * (0.189269f + t * 0.001308f)));
}

constexpr int kBins = 64;
constexpr int kCollect = 128;
constexpr int kSampleTiles = 8;   // moments from at least this many tiles per chunk
constexpr float kWinLo = 1.25f;   // histogram window around the predicted 64th score (sd)
constexpr float kWinHi = 0.75f;
constexpr int kCandRow = kCollect + 1;  // padded row strides (LDS bank spread)
constexpr int kHistRow = kBins + 5;  // 64 bins, 4 private overflow slots, 1 pad
enum RowMode : int { kModeAll = 0, kModeHist = 1, kModeFallback = 2 };

// Scores of one 64-key tile for the wave's 16 queries: acc[sub][v] is query
// (lane % 16) against key t0 + 16*sub + 4*(lane/16) + v, plus `init` (the
// kernels set it to the row's mean term b).
// bf16 and fp8 codes run on the bf16 MFMA (fp8 widened exactly to bf16 in
// registers), float32 codes on the f32 MFMA.
template <int RK, int ST>
struct MfmaScorer {
  static constexpr bool SBF = ST != kStF32;  // bf16 operands
  static constexpr bool F8 = ST == kStFp8;
  static constexpr int NKB = (SBF && RK >= 32) ? RK / 32 : 1;
  static constexpr int NKF = SBF ? 1 : RK / 4;
  static constexpr size_t TB = (size_t)kTile * RK * code_bytes<ST>();
  bf16x8_t zb[NKB];
  i16x4_t zb4;
  float zf[NKF];
  float init = 0.f;  // accumulator start (this lane's query column)

  // zs: this lane's query sketch row (RK floats, bf16 values for bf16 / fp8 codes)
  __device__ void load_operand(const float* zs, int g) {
    if constexpr (SBF) {
      if constexpr (RK == 16) {
        uint2 u;
        u.x = (__float_as_uint(zs[4 * g + 0]) >> 16) | (__float_as_uint(zs[4 * g + 1]) & 0xffff0000u);
        u.y = (__float_as_uint(zs[4 * g + 2]) >> 16) | (__float_as_uint(zs[4 * g + 3]) & 0xffff0000u);
        zb4 = as_i16x4(u);
      } else {
#pragma unroll
        for (int kk = 0; kk < NKB; ++kk) zb[kk] = as_bf16x8(pack_bf16x8(zs + 32 * kk + 8 * g));
      }
    } else {
#pragma unroll
      for (int m = 0; m < RK / 16; ++m)
#pragma unroll
        for (int e = 0; e < 4; ++e) zf[4 * m + e] = zs[4 * (g + 4 * m) + e];
    }
  }

  // zr: this lane's query sketch row as query_sketch_kernel writes it (RK
  // bf16 values for bf16 / fp8 codes, RK floats for float32 codes)
  __device__ void load_operand_row(const uint8_t* zr, int g) {
    if constexpr (SBF) {
      if constexpr (RK == 16) {
        zb4 = as_i16x4(*reinterpret_cast<const uint2*>(zr + 8 * g));
      } else {
#pragma unroll
        for (int kk = 0; kk < NKB; ++kk)
          zb[kk] = as_bf16x8(*reinterpret_cast<const uint4*>(zr + 2 * (32 * kk + 8 * g)));
      }
    } else {
#pragma unroll
      for (int m = 0; m < RK / 16; ++m) {
        const float4 v = *reinterpret_cast<const float4*>(zr + 4 * (4 * (g + 4 * m)));
        zf[4 * m] = v.x;
        zf[4 * m + 1] = v.y;
        zf[4 * m + 2] = v.z;
        zf[4 * m + 3] = v.w;
      }
    }
  }

  // raw operands of one tile: NL 16-byte loads per 16-key sub-block
  static constexpr int NL = SBF ? (RK == 16 ? 1 : RK / 32) : RK / 16;
  struct Raw {
    uint4 v[4][NL];
  };
  // the next tile is loaded while the current one is scored when its raw
  // operands fit in 32 registers
  static constexpr bool kPrefetch = 4 * NL <= 8;

  __device__ __forceinline__ void load(const uint8_t* tb, int qi, int g, Raw& r) const {
#pragma unroll
    for (int sub = 0; sub < 4; ++sub) {
      const int key = 16 * sub + qi;
      if constexpr (F8 && RK == 16) {  // dims 4g .. 4g+3: bytes 4g.. of piece 0
        const uint32_t raw = *reinterpret_cast<const uint32_t*>(tb + (size_t)key * 16 + 4 * g);
        r.v[sub][0] = uint4{raw, 0u, 0u, 0u};
      } else if constexpr (F8) {  // dims 32kk + 8g .. +7: piece 2kk + g/2, bytes 8(g%2)..
#pragma unroll
        for (int kk = 0; kk < NL; ++kk) {
          const uint2 raw = *reinterpret_cast<const uint2*>(
              tb + (size_t)(2 * kk + g / 2) * kTile * 16 + (size_t)key * 16 + (g % 2) * 8);
          r.v[sub][kk] = uint4{raw.x, raw.y, 0u, 0u};
        }
      } else if constexpr (SBF && RK == 16) {
        const uint2 raw = *reinterpret_cast<const uint2*>(tb + (size_t)(g / 2) * kTile * 16 +
                                                         (size_t)key * 16 + (g % 2) * 8);
        r.v[sub][0] = uint4{raw.x, raw.y, 0u, 0u};
      } else if constexpr (SBF) {
#pragma unroll
        for (int kk = 0; kk < NL; ++kk)
          r.v[sub][kk] = *reinterpret_cast<const uint4*>(tb + (size_t)(4 * kk + g) * kTile * 16 +
                                                         (size_t)key * 16);
      } else {
#pragma unroll
        for (int m = 0; m < NL; ++m)
          r.v[sub][m] = *reinterpret_cast<const uint4*>(tb + (size_t)(g + 4 * m) * kTile * 16 +
                                                        (size_t)key * 16);
      }
    }
  }

  __device__ __forceinline__ void mma(const Raw& r, f32x4_t acc[4]) const {
#pragma unroll
    for (int sub = 0; sub < 4; ++sub) {
      f32x4_t a = {init, init, init, init};
      if constexpr (F8 && RK == 16) {
        a = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(as_i16x4(e4m3x4_to_bf16(r.v[sub][0].x)), zb4,
                                                     a, 0, 0, 0);
      } else if constexpr (F8) {
#pragma unroll
        for (int kk = 0; kk < NL; ++kk) {
          const uint2 w0 = e4m3x4_to_bf16(r.v[sub][kk].x), w1 = e4m3x4_to_bf16(r.v[sub][kk].y);
          a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(uint4{w0.x, w0.y, w1.x, w1.y}),
                                                      zb[kk], a, 0, 0, 0);
        }
      } else if constexpr (SBF && RK == 16) {
        a = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(as_i16x4(uint2{r.v[sub][0].x, r.v[sub][0].y}),
                                                     zb4, a, 0, 0, 0);
      } else if constexpr (SBF) {
#pragma unroll
        for (int kk = 0; kk < NL; ++kk)
          a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(r.v[sub][kk]), zb[kk], a, 0, 0, 0);
      } else {
#pragma unroll
        for (int m = 0; m < NL; ++m) {
          const uint4 raw = r.v[sub][m];
          a = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(raw.x), zf[4 * m + 0], a, 0, 0, 0);
          a = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(raw.y), zf[4 * m + 1], a, 0, 0, 0);
          a = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(raw.z), zf[4 * m + 2], a, 0, 0, 0);
          a = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(raw.w), zf[4 * m + 3], a, 0, 0, 0);
        }
      }
      acc[sub] = a;
    }
  }

  // body(t0, acc) for the tiles t0 = t_beg, t_beg + step, ... < t_end
  template <class F>
  __device__ __forceinline__ void for_tiles(const uint8_t* hbase, int t_beg, int t_end, int step,
                                            int qi, int g, F&& body) const {
    if constexpr (kPrefetch) {
      // two register buffers taken in turn; the load past the last tile is
      // clamped to it (a valid, unused reload) so that no load is conditional
      if (t_beg >= t_end) return;
      const int last = t_beg + ((t_end - 1 - t_beg) / step) * step;
      auto at = [&](int t) { return hbase + (size_t)(min(t, last) / kTile) * TB; };
      Raw ra, rb;
      load(at(t_beg), qi, g, ra);
      for (int t0 = t_beg; t0 < t_end; t0 += 2 * step) {
        load(at(t0 + step), qi, g, rb);
        f32x4_t acc[4];
        mma(ra, acc);
        body(t0, acc);
        if (t0 + step >= t_end) break;
        load(at(t0 + 2 * step), qi, g, ra);
        mma(rb, acc);
        body(t0 + step, acc);
      }
    } else {
      for (int t0 = t_beg; t0 < t_end; t0 += step) {
        Raw cur;
        load(hbase + (size_t)(t0 / kTile) * TB, qi, g, cur);
        f32x4_t acc[4];
        mma(cur, acc);
        body(t0, acc);
      }
    }
  }

  // body(t0, acc) for every tile of [t_beg, t_end) in order, with the loads
  // of the next DEPTH - 1 tiles in flight while one is scored (a ring of
  // DEPTH register buffers) when a tile's operands fit in 32 registers;
  // otherwise as for_tiles.  Loads past the last tile are clamped to it.
  template <int DEPTH = 3, class F>
  __device__ __forceinline__ void for_tiles_deep(const uint8_t* hbase, int t_beg, int t_end,
                                                 int qi, int g, F&& body) const {
    if constexpr (kPrefetch) {
      if (t_beg >= t_end) return;
      const int last = t_beg + ((t_end - 1 - t_beg) / kTile) * kTile;
      auto at = [&](int t) { return hbase + (size_t)(min(t, last) / kTile) * TB; };
      Raw r[DEPTH];
#pragma unroll
      for (int d = 0; d + 1 < DEPTH; ++d) load(at(t_beg + d * kTile), qi, g, r[d]);
      for (int t0 = t_beg;; t0 += DEPTH * kTile) {
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
          const int t = t0 + d * kTile;
          load(at(t + (DEPTH - 1) * kTile), qi, g, r[(d + DEPTH - 1) % DEPTH]);
          f32x4_t acc[4];
          mma(r[d], acc);
          body(t, acc);
          if (t + kTile >= t_end) return;
        }
      }
    } else {
      for_tiles(hbase, t_beg, t_end, kTile, qi, g, body);
    }
  }
};

// The query sketch of a wave's 16 rows (lane (qi, g) = lane % 16, lane / 16)
// on the f32 MFMA: D[m][qi] = sum_c B_q[c][m] q[qi][c] with lane group g
// feeding dims c = 4s + g, rounded to bf16 for bf16 and fp8 codes and staged
// through zs (16 x RK floats of LDS) into the scorer's operand.  Returns
// b = q . mu of row qi (the same in its four lanes).  qr: row qi's query (any
// valid row when !row_ok, whose query counts as zero).
template <int RK, int ST>
__device__ __forceinline__ float mfma_query_sketch(const float* __restrict__ qr, bool row_ok,
                                                   const float* __restrict__ bq,
                                                   const float* __restrict__ mr, float* zs, int qi,
                                                   int g, MfmaScorer<RK, ST>& sc) {
  constexpr int D = saki::kHeadDim;
  f32x4_t za[RK / 16];
#pragma unroll
  for (int mb = 0; mb < RK / 16; ++mb) za[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float bp = 0.f;
  // the loads of SB steps are issued together, then their products taken
  constexpr int SB = RK <= 32 ? 16 : RK <= 64 ? 8 : 4;
#pragma unroll 1
  for (int s0 = 0; s0 < D / 4; s0 += SB) {
    float qa[SB], ma[SB], ba[SB][RK / 16];
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      const int c = 4 * (s0 + u) + g;
      qa[u] = qr[c];
      ma[u] = mr[c];
#pragma unroll
      for (int mb = 0; mb < RK / 16; ++mb) ba[u][mb] = bq[c * RK + 16 * mb + qi];
    }
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      const float qv = row_ok ? qa[u] : 0.f;
      bp = fmaf(qv, ma[u], bp);
#pragma unroll
      for (int mb = 0; mb < RK / 16; ++mb)
        za[mb] = __builtin_amdgcn_mfma_f32_16x16x4f32(ba[u][mb], qv, za[mb], 0, 0, 0);
    }
  }
  const float b = sum_lane_groups(bp);
#pragma unroll
  for (int mb = 0; mb < RK / 16; ++mb)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const float zv = za[mb][v];
      zs[qi * RK + 16 * mb + 4 * g + v] = ST != kStF32 ? bf16_round(zv) : zv;
    }
  wave_lds_sync();
  sc.load_operand(zs + qi * RK, g);
  wave_lds_sync();
  return b;
}

// ---------------------------------------------------------------- query sketches of a batch of rows

// query_sketch_kernel: z = B_q^T q and b = q . mu (equation (5): the query
// side of the factored score) of every row, written once so that the
// two-pass scoring kernel loads each wave's 16 rows as one contiguous block.
// z is rounded to bf16 for bf16 and fp8 codes (the MFMA operand) and kept in
// float32 for float32 codes; row layout zq[(bh * Q + i) * RK + m], b[bh * Q + i].
// The f32 MFMA forms D[m][qi] = sum_c B_q[c][m] q[qi][c]: lane (qi, g) loads
// q[qi][16j + 4g .. 16j + 4g + 3] for j = 0..7 as float4 (each row read as
// 64-byte runs) and feeds dims c = 16j + 4g + e at step 4j + e.  B_q of the
// head waits in LDS in that operand order, one float4 per (j, mb) and lane.
// grid: 1-D, work-group (bh, part) covers rows [part * kQsRows, ...) of (b, h).
constexpr int kQsWaves = 4;
constexpr int kQsRows = 1024;

template <int RK, int ST>
__global__ __launch_bounds__(kQsWaves * kWave) void query_sketch_kernel(
    const float* __restrict__ q, const float* __restrict__ Bq, const float* __restrict__ mu,
    int Q, int H_q, int H_kv, int n_bh, int parts, uint8_t* __restrict__ zq,
    float* __restrict__ bout) {
  constexpr int D = saki::kHeadDim;
  constexpr int MB = RK / 16;
  __shared__ __align__(16) float bl[D * RK];
  const long long lb = xcd_logical_block((long long)n_bh * parts);
  if (lb < 0) return;
  const size_t bh = (size_t)(lb / parts);
  const int part = (int)(lb % parts);
  const int h = (int)(bh % H_q);
  const int gkv = h / (H_q / H_kv);
  // B_q[h] (row-major D x RK) -> bl[((j * MB + mb) * 64 + 16 g + qi) * 4 + e]
  // = B_q[16j + 4g + e][16mb + qi]
  const float* bsrc = Bq + (size_t)h * D * RK;
  for (int i = threadIdx.x; i < D * RK; i += kQsWaves * kWave) {
    const int c = i / RK, m = i % RK;
    bl[(((c / 16) * MB + m / 16) * 64 + 16 * ((c % 16) / 4) + m % 16) * 4 + c % 4] = bsrc[i];
  }
  __syncthreads();
  const int wave = threadIdx.x / kWave, lane = lane_id();
  const int qi = lane % 16, g = lane / 16;
  const float* mr = mu + (size_t)gkv * D;
  float4 mv[8];  // this lane's dims of mu
#pragma unroll
  for (int j = 0; j < 8; ++j) mv[j] = *reinterpret_cast<const float4*>(mr + 16 * j + 4 * g);
  const int r_end = min(Q, (part + 1) * kQsRows);
  for (int row0 = part * kQsRows + wave * kMR; row0 < r_end; row0 += kQsWaves * kMR) {
    const int row = row0 + qi;
    const bool ok = row < r_end;
    const float* qr = q + (bh * Q + (ok ? row : row0)) * D;
    float4 qv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      qv[j] = *reinterpret_cast<const float4*>(qr + 16 * j + 4 * g);
      if (!ok) qv[j] = float4{0.f, 0.f, 0.f, 0.f};
    }
    float bp = 0.f;
    f32x4_t za[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) za[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      bp = fmaf(qv[j].x, mv[j].x, bp);
      bp = fmaf(qv[j].y, mv[j].y, bp);
      bp = fmaf(qv[j].z, mv[j].z, bp);
      bp = fmaf(qv[j].w, mv[j].w, bp);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const float4 a = *reinterpret_cast<const float4*>(bl + ((j * MB + mb) * 64 + lane) * 4);
        za[mb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, qv[j].x, za[mb], 0, 0, 0);
        za[mb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, qv[j].y, za[mb], 0, 0, 0);
        za[mb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, qv[j].z, za[mb], 0, 0, 0);
        za[mb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, qv[j].w, za[mb], 0, 0, 0);
      }
    }
    const float b = sum_lane_groups(bp);
    if (!ok) continue;
    const size_t base = (bh * Q + row) * RK;
    // lane (qi, g) holds z[row][16mb + 4g + v], v = 0..3
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      if constexpr (ST != kStF32) {
        const uint2 u{bf16_bits(za[mb][0]) | (bf16_bits(za[mb][1]) << 16),
                      bf16_bits(za[mb][2]) | (bf16_bits(za[mb][3]) << 16)};
        *reinterpret_cast<uint2*>(zq + (base + 16 * mb + 4 * g) * 2) = u;
      } else {
        *reinterpret_cast<float4*>(zq + (base + 16 * mb + 4 * g) * 4) =
            float4{za[mb][0], za[mb][1], za[mb][2], za[mb][3]};
      }
    }
    if (g == 0) bout[bh * Q + row] = b;
  }
}

// ---------------------------------------------------------------- sketch scoring, MFMA, block-maximum gate

// score_batch_kernel: one wave per work-group (its LDS is released the moment
// it ends, where a wave of a larger work-group would hold its slot until the
// slowest of its siblings ends), each with a block of 16 query rows and that
// block's keys of one chunk (at most 4,096 keys), and the exact top-64 per row
// in two passes over the codes (the MFMA recomputes the scores in the second).  Rows are ranked by s' = z . c: b is
// the same for all keys of a row and is added to the 64 kept scores.
//   A. each lane records the maxima of its keys in blocks of 8, 4, 2 or 1
//      keys, the size set by the wave's longest row (at least 2,048, 1,024,
//      512 keys, or fewer), so that a row of at least about 256 keys has
//      about 256 blocks or more and the rows of a wave below 512 keys have
//      one block per key.  A maximum is stored as the top 16 bits of its
//      ordered float32 bits, which rounds it down.
//   threshold: per row, a histogram of the stored maxima over 64 equal bins
//      of score around the predicted 64th largest (from their mean and
//      spread and a normal quantile; moved above or below when the crossing
//      falls outside) gives tau, the lower edge of the bin below the highest
//      bin whose count from the top reaches 64.  At least 64 blocks then
//      have a maximum >= tau, so at least 64 keys score >= tau and all of
//      the row's top-64 do; with 256 blocks or more about 64-90 keys pass.
//      A row with fewer than 64 blocks keeps every key.
//   B. every key that scores >= tau goes to its lane's candidate slots (39
//      per lane usable, 156 per row), and the row's count is checked to be
//      >= 64.
// The candidates are then sorted by a bitonic network that holds 16 entries
// per lane, and the best 64 are kept.  A row whose candidates overflow its
// slots (many equal scores, or rows of very different lengths in one wave)
// or fall short sends its wave to the online selection of saki_topk.h.

constexpr int kBWaves = saki::kBatchWaves;  // independent waves per work-group
constexpr int kBEnt = 512;                 // block-maximum entries per row
constexpr int kBBins = 64;                 // histogram bins per row
constexpr int kBSlots = 40;                // candidate slots per lane
constexpr int kBDepth = 3;                 // code tiles whose loads are in flight, plus one
constexpr int kBWaveBytes = kMR * 4 * kBSlots * 8;  // 20 KiB of LDS per wave
static_assert(saki::kBatchMaxChunk / 8 <= kBEnt, "a chunk's 8-key blocks fit");
static_assert(kMR * kBEnt * 2 + kMR * kBBins * 4 <= kBWaveBytes, "entries and bins fit");
static_assert(kMR * kTile * 4 + 2 * (kMR / 2) * kList * 8 <= kBWaveBytes, "fallback fits");

// Top 16 bits of the ordered float32 bits: rounds down, finite values map to
// 0x0080 and above, and -inf (a masked key) to 0.
__device__ __forceinline__ uint32_t ord16(float x) {
  return x == -INFINITY ? 0u : (ord_f32(x) >> 16);
}
// The float an entry stands for (at most the maximum it was taken from).
__device__ __forceinline__ float unord16(uint32_t v) { return unord_f32(v << 16); }
// ord16(a) | ord16(b) << 16 for finite a and b.
__device__ __forceinline__ uint32_t pack_ord16(float a, float b) {
  const uint32_t ua = __float_as_uint(a), ub = __float_as_uint(b);
  const uint32_t oa = ua ^ ((uint32_t)((int32_t)ua >> 31) | 0x80000000u);
  const uint32_t ob = ub ^ ((uint32_t)((int32_t)ub >> 31) | 0x80000000u);
  return __builtin_amdgcn_perm(ob, oa, 0x07060302u);  // bytes 2, 3 of oa, then of ob
}

// Bitonic sort of one row's 64 entries held 16 per lane by the row's four
// lanes (lane groups g = lane / 16): entry e = 16 g + i is x[i] of lane group
// g.  Leaves the entries in descending order of e.
template <class KO>
__device__ __forceinline__ void sort64_x16(typename KO::K (&x)[16], int g) {
  using K = typename KO::K;
#pragma unroll
  for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
    for (int m = k >> 1; m > 0; m >>= 1) {
      if (m >= 16) {  // partner in lane group g ^ (m / 16): lane xor m
        const bool lower = (g & (m >> 4)) == 0;
        const bool desc = k == 64 || (g & (k >> 4)) == 0;
        const bool keep_better = lower == desc;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const K o = KO::shfl_xor(x[i], m);
          x[i] = KO::sel(KO::gt(x[i], o) == keep_better, x[i], o);
        }
      } else {  // partner in the same lane
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          if (i & m) continue;
          const int j = i | m;
          const bool desc = k >= 64 ? true : k >= 16 ? (g & (k >> 4)) == 0 : (i & k) == 0;
          const K a = x[i], b = x[j];
          const bool sw = KO::gt(a, b) != desc;  // the lower position takes the better when descending
          x[i] = KO::sel(sw, b, a);
          x[j] = KO::sel(sw, a, b);
        }
      }
    }
  }
}

// x <- the best 64 of x and y (both sorted descending as left by sort64_x16).
template <class KO>
__device__ __forceinline__ void merge64_x16(typename KO::K (&x)[16], const typename KO::K (&y)[16],
                                            int g) {
  using K = typename KO::K;
  // entry e against y's entry 63 - e = 16 (3 - g) + (15 - i): lane group g ^ 3
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const K r = KO::shfl_xor(KO::shfl_xor(y[15 - i], 16), 32);
    x[i] = KO::sel(KO::gt(r, x[i]), r, x[i]);
  }
  // x is now bitonic: half-cleaners, all descending
#pragma unroll
  for (int m = 32; m >= 16; m >>= 1) {
    const bool lower = (g & (m >> 4)) == 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const K o = KO::shfl_xor(x[i], m);
      x[i] = KO::sel(KO::gt(x[i], o) == lower, x[i], o);
    }
  }
#pragma unroll
  for (int m = 8; m > 0; m >>= 1) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (i & m) continue;
      const int j = i | m;
      const K a = x[i], b = x[j];
      const bool sw = KO::gt(b, a);
      x[i] = KO::sel(sw, b, a);
      x[j] = KO::sel(sw, a, b);
    }
  }
}

// ---- 32-bit keys, 64 per row held 16 per lane as in sort64_x16

__device__ __forceinline__ uint32_t umax32(uint32_t a, uint32_t b) { return a > b ? a : b; }
__device__ __forceinline__ uint32_t umin32(uint32_t a, uint32_t b) { return a < b ? a : b; }
// a takes the larger key, b the smaller
__device__ __forceinline__ void cx_u32(uint32_t& a, uint32_t& b) {
  const uint32_t hi = umax32(a, b);
  b = umin32(a, b);
  a = hi;
}
// Compare-exchange of entry X of lane groups g and g ^ (M / 16), and the same
// for entry Y; the lower lane group keeps the larger key.  The first permlane
// swap hands every lane one such pair (of X in half of the lane groups, of Y
// in the others), and the second sends the larger and the smaller back.
template <int M>
__device__ __forceinline__ void cx_rows_u32(uint32_t& X, uint32_t& Y) {
  if constexpr (M == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(X, Y, false, false);
    const auto t = __builtin_amdgcn_permlane16_swap(umax32(r[0], r[1]), umin32(r[0], r[1]), false, false);
    X = t[0];
    Y = t[1];
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(X, Y, false, false);
    const auto t = __builtin_amdgcn_permlane32_swap(umax32(r[0], r[1]), umin32(r[0], r[1]), false, false);
    X = t[0];
    Y = t[1];
  }
}
// Stages m = 8, 4, 2, 1 of a descending bitonic merge inside each lane.
__device__ __forceinline__ void lane_merge_desc_u32(uint32_t (&x)[16]) {
#pragma unroll
  for (int m = 8; m > 0; m >>= 1)
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (!(i & m)) cx_u32(x[i], x[i | m]);
}
// Bitonic sort of one row's 64 keys into descending order of e = 16 g + i.
// Blocks whose direction depends on the lane group (levels 16 and 32) are
// sorted as complemented keys, so every stage there is descending.
__device__ __forceinline__ void sort64_u32(uint32_t (&x)[16], int g) {
#pragma unroll
  for (int k = 2; k <= 8; k <<= 1)
#pragma unroll
    for (int m = k >> 1; m > 0; m >>= 1)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        if (i & m) continue;
        if ((i & k) == 0)
          cx_u32(x[i], x[i | m]);
        else
          cx_u32(x[i | m], x[i]);
      }
  const uint32_t c1 = (g & 1) ? ~0u : 0u, c2 = (g & 2) ? ~0u : 0u;
#pragma unroll
  for (int i = 0; i < 16; ++i) x[i] ^= c1;
  lane_merge_desc_u32(x);  // level 16
#pragma unroll
  for (int i = 0; i < 16; ++i) x[i] ^= c1 ^ c2;
#pragma unroll
  for (int i = 0; i < 16; i += 2) cx_rows_u32<16>(x[i], x[i + 1]);  // level 32
  lane_merge_desc_u32(x);
#pragma unroll
  for (int i = 0; i < 16; ++i) x[i] ^= c2;
#pragma unroll
  for (int i = 0; i < 16; i += 2) cx_rows_u32<32>(x[i], x[i + 1]);  // level 64
#pragma unroll
  for (int i = 0; i < 16; i += 2) cx_rows_u32<16>(x[i], x[i + 1]);
  lane_merge_desc_u32(x);
}
// x <- the best 64 of x (descending) and y (ascending); dmax <- the largest
// key left out so far.  The elementwise maxima form a bitonic sequence.
__device__ __forceinline__ void merge64_u32(uint32_t (&x)[16], const uint32_t (&y)[16],
                                            uint32_t& dmax) {
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    dmax = umax32(dmax, umin32(x[i], y[i]));
    x[i] = umax32(x[i], y[i]);
  }
#pragma unroll
  for (int i = 0; i < 16; i += 2) cx_rows_u32<32>(x[i], x[i + 1]);
#pragma unroll
  for (int i = 0; i < 16; i += 2) cx_rows_u32<16>(x[i], x[i + 1]);
  lane_merge_desc_u32(x);
}

// grid: 1-D, 8 * ceil(groups * n_chunks * n_bh / 8) work-groups of kBWaves
// waves; work-group (bh, chunk, group) takes the 16-row blocks kBWaves * group
// .. kBWaves * group + kBWaves - 1 of (sequence, head) bh, the longest causal
// rows first.
template <int RK, int ST>
__global__ __launch_bounds__(kBWaves * kWave) void score_batch_kernel(
    const uint8_t* __restrict__ index, int n_tiles, int N_valid, int Q,
    const int* __restrict__ q_pos, const uint8_t* __restrict__ zq,
    const float* __restrict__ zb, int H_q, int gq, int n_bh, int groups, int chunk,
    int n_chunks, int k, int* __restrict__ top_idx, float* __restrict__ top_score,
    uint64_t* __restrict__ part) {
  constexpr int D = saki::kHeadDim;
  using KO = KeysF32;
  using K = uint64_t;
  using Scorer = MfmaScorer<RK, ST>;
  __shared__ __align__(16) uint8_t lds_mem[kBWaves][kBWaveBytes];
  const int wave = threadIdx.x / kWave, lane = lane_id();
  const long long lb = xcd_logical_block((long long)groups * n_chunks * n_bh);
  if (lb < 0) return;
  const int gb = groups - 1 - (int)(lb % groups);
  const int ch = (int)((lb / groups) % n_chunks);
  const size_t bh = (size_t)(lb / ((long long)groups * n_chunks));
  const int h = (int)(bh % H_q);
  const int row0 = (gb * kBWaves + wave) * kMR;
  if (row0 >= Q) return;  // the waves never synchronise with each other
  const int qi = lane % 16, g = lane / 16;
  const int my_row = row0 + qi;
  const bool row_ok = my_row < Q;
  const int my_lim = row_limit(my_row, Q, N_valid, q_pos);  // 0 for rows past Q
  const int kmax = wave_max_i(my_lim);
  const int kmin = wave_min_i(my_lim);
  const int kbeg = ch * chunk;
  const int kend = min(kbeg + chunk, kmax);
  uint8_t* wl = lds_mem[wave];

  // ---- query sketch, formed by query_sketch_kernel.  b = q . mu is the same
  // for every key of a row, so the selection ranks s' = z . c (accumulators
  // starting at zero) and b is added to the 64 scores that are kept.
  Scorer sc;
  const size_t zrow = bh * Q + (row_ok ? my_row : row0);
  sc.load_operand_row(zq + zrow * RK * (ST != kStF32 ? 2 : 4), g);
  const float my_b = zb[zrow];
  const size_t code_set = (bh / H_q) * (H_q / gq) + h / gq;
  const uint8_t* hbase = index + code_set * n_tiles * Scorer::TB;

  // keys past a row's limit score -inf (tiles crossing some row's limit only)
  auto mask_tile = [&](int t0, f32x4_t* acc) {
    if (t0 + kTile > kmin) {
#pragma unroll
      for (int sub = 0; sub < 4; ++sub)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (t0 + 16 * sub + 4 * g + v >= my_lim) acc[sub][v] = -INFINITY;
    }
  };

  // ---- pass A: block maxima of this lane's keys
  const int n_row = max(0, min(my_lim, kend) - kbeg);
  const int row_tiles = (n_row + kTile - 1) / kTile;
  // entries of one lane per tile: 2, 4, 8 or 16 blocks of 8, 4, 2 or 1 keys,
  // by the wave's longest row (kend - kbeg keys), so that no row has more
  // than kBEnt entries
  const int n_wave = kend - kbeg;
  const int lane_ent = n_wave >= 2048 ? 2 : n_wave >= 1024 ? 4 : n_wave >= 512 ? 8 : 16;
  // row qi's entries and histogram bins have their 16-byte groups permuted
  // (word offset xor 4 qi), so that the rows' accesses spread over the banks
  uint32_t* ent = reinterpret_cast<uint32_t*>(wl) + qi * (kBEnt / 2);
  const int sw = 4 * qi;
  float bsum = 0.f, bsq = 0.f, bmax = -INFINITY, bmin = INFINITY, bcnt = 0.f;
  auto stat = [&](float x) {  // x: a block maximum (-inf: no key of the row)
    const bool ok = x != -INFINITY;
    const float y = ok ? x : 0.f;
    bcnt += ok ? 1.f : 0.f;
    bsum += y;
    bsq = fmaf(y, y, bsq);
    bmax = vmax(bmax, x);
    bmin = ok ? vmin(bmin, x) : bmin;
  };
  sc.template for_tiles_deep<kBDepth>(hbase, kbeg, kend, qi, g, [&](int t0, f32x4_t* acc) {
    const int tl = (t0 - kbeg) / kTile;
    const int wo = (tl * 4 * lane_ent + g * lane_ent) / 2;  // this lane's first word
    if (t0 + kTile <= kmin && lane_ent <= 4) {
      // every key of the tile lies below every row's limit: no -inf
      if (lane_ent == 2) {
        const float a = vmax(vmax(vmax(acc[0][0], acc[0][1]), vmax(acc[0][2], acc[0][3])),
                             vmax(vmax(acc[1][0], acc[1][1]), vmax(acc[1][2], acc[1][3])));
        const float b = vmax(vmax(vmax(acc[2][0], acc[2][1]), vmax(acc[2][2], acc[2][3])),
                             vmax(vmax(acc[3][0], acc[3][1]), vmax(acc[3][2], acc[3][3])));
        ent[wo ^ sw] = pack_ord16(a, b);
        bsum += a + b;
        bsq = fmaf(a, a, fmaf(b, b, bsq));
        bmax = vmax(bmax, vmax(a, b));
        bmin = vmin(bmin, vmin(a, b));
        bcnt += 2.f;
      } else {
        float m4[4];
#pragma unroll
        for (int sub = 0; sub < 4; ++sub)
          m4[sub] = vmax(vmax(acc[sub][0], acc[sub][1]), vmax(acc[sub][2], acc[sub][3]));
        *reinterpret_cast<uint2*>(ent + (wo ^ sw)) = uint2{pack_ord16(m4[0], m4[1]), pack_ord16(m4[2], m4[3])};
        bsum += (m4[0] + m4[1]) + (m4[2] + m4[3]);
        bsq = fmaf(m4[0], m4[0], fmaf(m4[1], m4[1], fmaf(m4[2], m4[2], fmaf(m4[3], m4[3], bsq))));
        bmax = vmax(vmax(bmax, vmax(m4[0], m4[1])), vmax(m4[2], m4[3]));
        bmin = vmin(vmin(bmin, vmin(m4[0], m4[1])), vmin(m4[2], m4[3]));
        bcnt += 4.f;
      }
      return;
    }
    mask_tile(t0, acc);
    if (tl >= row_tiles) return;  // nothing of this row: no entries
    float m2[8];  // maxima of the pairs (sub, v = 0..1), (sub, v = 2..3)
#pragma unroll
    for (int sub = 0; sub < 4; ++sub) {
      m2[2 * sub] = vmax(acc[sub][0], acc[sub][1]);
      m2[2 * sub + 1] = vmax(acc[sub][2], acc[sub][3]);
    }
    if (lane_ent == 2) {
      const float a = vmax(vmax(m2[0], m2[1]), vmax(m2[2], m2[3]));
      const float b = vmax(vmax(m2[4], m2[5]), vmax(m2[6], m2[7]));
      ent[wo ^ sw] = ord16(a) | (ord16(b) << 16);
      stat(a);
      stat(b);
    } else if (lane_ent == 4) {
      uint32_t u[4];
#pragma unroll
      for (int sub = 0; sub < 4; ++sub) {
        const float m4 = vmax(m2[2 * sub], m2[2 * sub + 1]);
        u[sub] = ord16(m4);
        stat(m4);
      }
      *reinterpret_cast<uint2*>(ent + (wo ^ sw)) = uint2{u[0] | (u[1] << 16), u[2] | (u[3] << 16)};
    } else if (lane_ent == 8) {
      uint32_t u[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        u[j] = ord16(m2[j]);
        stat(m2[j]);
      }
      *reinterpret_cast<uint4*>(ent + (wo ^ sw)) =
          uint4{u[0] | (u[1] << 16), u[2] | (u[3] << 16), u[4] | (u[5] << 16), u[6] | (u[7] << 16)};
    } else {
      uint32_t u[16];
#pragma unroll
      for (int sub = 0; sub < 4; ++sub)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          u[4 * sub + v] = ord16(acc[sub][v]);
          stat(acc[sub][v]);
        }
      *reinterpret_cast<uint4*>(ent + (wo ^ sw)) =
          uint4{u[0] | (u[1] << 16), u[2] | (u[3] << 16), u[4] | (u[5] << 16), u[6] | (u[7] << 16)};
      *reinterpret_cast<uint4*>(ent + ((wo + 4) ^ sw)) = uint4{u[8] | (u[9] << 16), u[10] | (u[11] << 16),
                                                             u[12] | (u[13] << 16), u[14] | (u[15] << 16)};
    }
  });
  wave_lds_sync();

  // ---- threshold per row
  bsum = sum_lane_groups(bsum);
  bsq = sum_lane_groups(bsq);
  bcnt = sum_lane_groups(bcnt);
  bmax = fmaxf(bmax, xor_shfl_f32(bmax, 16));
  bmax = fmaxf(bmax, xor_shfl_f32(bmax, 32));
  bmin = fminf(bmin, xor_shfl_f32(bmin, 16));
  bmin = fminf(bmin, xor_shfl_f32(bmin, 32));
  const int n_ent = row_tiles * 4 * lane_ent;
  float tau = -FLT_MAX;  // rows with fewer than 64 blocks keep every key
  bool done = bcnt < (float)kList;
  float lo = 0.f, hi = 0.f;
  if (!done) {
    const float mean = bsum / bcnt;
    const float sd = sqrtf(fmaxf(bsq / bcnt - mean * mean, 0.f));
    const float tail = (float)kList / bcnt;  // in (0, 1]
    const float zq = tail <= 0.5f ? normal_upper_quantile(tail)
                                  : (tail < 1.f ? -normal_upper_quantile(1.f - tail) : -4.f);
    const float pred = mean + sd * zq;  // predicted 64th largest maximum
    lo = fmaxf(pred - 1.5f * sd, bmin);
    hi = fminf(pred + 0.5f * sd, bmax);
    if (!(hi > lo)) {  // all maxima (nearly) equal
      tau = bmin;
      done = true;
    }
  }
  uint32_t* hist = reinterpret_cast<uint32_t*>(wl + kMR * kBEnt * 2) + qi * kBBins;  // bin b at word b ^ sw
  for (int round = 0; __ballot(!done) != 0; ++round) {
#pragma unroll
    for (int u = 0; u < 4; ++u)
      *reinterpret_cast<uint4*>(hist + ((16 * g + 4 * u) ^ sw)) = uint4{0u, 0u, 0u, 0u};
    wave_lds_sync();
    const float inv_w = (float)(kBBins - 1) / (hi - lo);  // bins 0..62 over [lo, hi), 63 above
    const float off = -lo * inv_w;
    if (!done) {
      // an entry (in the top 16 bits of o) counts in bin (its value - lo) * inv_w,
      // cut to 63, unless that is below 0; an empty entry reads as NaN and
      // does not count
      auto count = [&](uint32_t o) {
        const uint32_t bits = o ^ (~(uint32_t)((int32_t)o >> 31) | 0x80000000u);
        const float x = fmaf(__uint_as_float(bits), inv_w, off);
        const int b = min((int)x, kBBins - 1);
        if (x >= 0.f) atomicAdd(&hist[b ^ sw], 1u);
      };
#pragma unroll 2
      for (int e0 = 8 * g; e0 < n_ent; e0 += 32) {  // this lane's quarter of the row's entries
        const uint4 w = *reinterpret_cast<const uint4*>(ent + ((e0 / 2) ^ sw));
        const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          count(ww[u] << 16);
          count(ww[u] & 0xffff0000u);
        }
      }
    }
    wave_lds_sync();
    // bins 16 g .. 16 g + 15 of this lane's row: counts from the top
    uint32_t c[16];
    {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint4 t = *reinterpret_cast<const uint4*>(hist + ((16 * g + 4 * u) ^ sw));
        c[4 * u] = t.x;
        c[4 * u + 1] = t.y;
        c[4 * u + 2] = t.z;
        c[4 * u + 3] = t.w;
      }
    }
    uint32_t run = 0;
#pragma unroll
    for (int i = 15; i >= 0; --i) {
      run += c[i];
      c[i] = run;
    }
    const uint32_t t1 = xor_shfl_u32(run, 16), t2 = xor_shfl_u32(run, 32), t3 = xor_shfl_u32(t1, 32);
    // totals of the lane groups above g (groups g ^ 1, g ^ 2, g ^ 3 hold t1, t2, t3)
    const uint32_t above = g == 0 ? t1 + t2 + t3 : g == 1 ? t2 + t3 : g == 2 ? t1 : 0u;
    int n_ge = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) n_ge += (c[i] + above >= (uint32_t)kList) ? 1 : 0;
    int b = n_ge > 0 ? 16 * g + n_ge - 1 : -1;
    b = max(b, (int)xor_shfl_u32((uint32_t)b, 16));
    b = max(b, (int)xor_shfl_u32((uint32_t)b, 32));
    if (!done) {
      const float w = (hi - lo) / (float)(kBBins - 1);
      if (round >= 3) {  // no usable window: keep every key (the count check decides)
        done = true;
      } else if (b < 0) {  // the 64th largest maximum lies below the window
        hi = lo;
        lo = bmin;
        done = !(hi > lo);
      } else if (b == kBBins - 1 && hi < bmax) {  // or above it
        lo = hi;
        hi = bmax;
      } else {
        // one bin lower than the crossing: rounding in the bin index never
        // puts a maximum below tau
        tau = lo + (float)(b - 1) * w;
        done = true;
      }
    }
    wave_lds_sync();
  }

  // ---- pass B: candidates, every key scoring >= tau
  // Slot j of a lane holds a score bits at word 128 j + lane and its key at
  // word 128 j + 64 + lane (so that the lanes' writes spread over the banks
  // and a pair is one two-address write).  Every score is written to the
  // lane's next free slot and the pointer moves on only past one >= tau, so
  // no lane branches; a lane whose count reaches the last slot keeps
  // counting and overwrites it (and the wave then takes the fallback below).
  uint32_t* const cw = reinterpret_cast<uint32_t*>(wl) + lane;
  uint32_t* wp = cw;
  int cnt = 0;
  sc.template for_tiles_deep<kBDepth>(hbase, kbeg, kend, qi, g, [&](int t0, f32x4_t* acc) {
    mask_tile(t0, acc);
    const uint32_t kb = (uint32_t)(t0 + 4 * g);
    if (__ballot(cnt > kBSlots - 16) == 0) {  // room for the whole tile in every lane
#pragma unroll
      for (int sub = 0; sub < 4; ++sub)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          wp[0] = __float_as_uint(acc[sub][v]);
          wp[kWave] = kb + (uint32_t)(16 * sub + v);
          wp += acc[sub][v] >= tau ? 2 * kWave : 0;
        }
      cnt = (int)(wp - cw) / (2 * kWave);
    } else {
#pragma unroll
      for (int sub = 0; sub < 4; ++sub)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          uint32_t* sp = cw + 2 * kWave * min(cnt, kBSlots - 1);
          sp[0] = __float_as_uint(acc[sub][v]);
          sp[kWave] = kb + (uint32_t)(16 * sub + v);
          cnt += acc[sub][v] >= tau ? 1 : 0;
        }
      wp = cw + 2 * kWave * min(cnt, kBSlots - 1);
    }
  });

  // the row's candidates: at least 64 unless every key of the row is one
  int row_cnt = cnt + (int)xor_shfl_u32((uint32_t)cnt, 16);
  row_cnt += (int)xor_shfl_u32((uint32_t)row_cnt, 32);
  const bool short_row = tau > -FLT_MAX && row_cnt < kList;
  if (__ballot(cnt >= kBSlots || short_row) == 0) {
    // ---- sort the candidates, keep the best 64
    wave_lds_sync();
    const uint32_t* const wbase = cw - lane;  // word 0 of the wave's slots
    // 32-bit keys: the top 24 bits of the ordered score s', then the
    // candidate's id 4 slot + g (0 past the lane's count)
    auto key32 = [&](int j) -> uint32_t {
      const uint32_t sb = cw[2 * kWave * min(j, kBSlots - 1)];
      const uint32_t o = sb ^ ((uint32_t)((int32_t)sb >> 31) | 0x80000000u);
      return j < cnt ? (o & 0xffffff00u) | (uint32_t)(4 * j + g) : 0u;
    };
    uint32_t x32[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) x32[i] = key32(i);
    sort64_u32(x32, g);
    uint32_t dmax = 0u;  // the best key left out
    // the slots past the first 16 of each lane, 16 at a time, sorted
    // ascending (as complemented keys) and merged
#pragma unroll 1
    for (int set = 1; 16 * set < kBSlots && __ballot(cnt > 16 * set) != 0; ++set) {
      uint32_t y[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) y[i] = ~key32(16 * set + i);
      sort64_u32(y, g);
#pragma unroll
      for (int i = 0; i < 16; ++i) y[i] = ~y[i];
      merge64_u32(x32, y, dmax);
    }
    // the kept set is certain unless the 64th kept key and the best one left
    // out share their top 24 bits
    dmax = umax32(dmax, xor_shfl_u32(dmax, 16));
    dmax = umax32(dmax, xor_shfl_u32(dmax, 32));
    // entry 63 of the row (x32[15] of lane group 3) in all four lanes; every
    // lane takes part in both swaps
    const uint32_t s32 = xor_shfl_u32(x32[15], 32);
    const uint32_t t32 = (g & 2) ? x32[15] : s32;
    const uint32_t s16 = xor_shfl_u32(t32, 16);
    const uint32_t k64 = (g & 1) ? t32 : s16;
    const bool unsure = dmax != 0u && (dmax >> 8) == (k64 >> 8);
    K x[16];
    if (__ballot(unsure) == 0) {
      // the kept entries as exact keys of (s' + b, index), in key order up to
      // runs of equal top 24 bits; two odd-even transposition steps put runs
      // of two in order (what is left is found below)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const uint32_t id = x32[i] & 0xffu;
        const uint32_t* c = wbase + 2 * kWave * (id >> 2) + 16 * (id & 3) + qi;
        x[i] = x32[i] == 0u ? KO::pad() : KO::make(__uint_as_float(c[0]) + my_b, (int)c[kWave]);
      }
      auto cx64 = [](K& a, K& b2) {
        const bool sw = KO::gt(b2, a);
        const K t = a;
        a = KO::sel(sw, b2, a);
        b2 = KO::sel(sw, t, b2);
      };
#pragma unroll
      for (int i = 0; i < 16; i += 2) cx64(x[i], x[i + 1]);
#pragma unroll
      for (int i = 1; i < 15; i += 2) cx64(x[i], x[i + 1]);
      {  // entries 16 g + 15 and 16 (g + 1), held by lanes 16 apart
        const K nxt = ((uint64_t)(uint32_t)__shfl_down((int)(uint32_t)(x[0] >> 32), 16, kWave) << 32) |
                      (uint32_t)__shfl_down((int)(uint32_t)x[0], 16, kWave);
        const K prv = ((uint64_t)(uint32_t)__shfl_up((int)(uint32_t)(x[15] >> 32), 16, kWave) << 32) |
                      (uint32_t)__shfl_up((int)(uint32_t)x[15], 16, kWave);
        if (g < 3 && KO::gt(nxt, x[15])) x[15] = nxt;
        if (g > 0 && KO::gt(x[0], prv)) x[0] = prv;
      }
    } else {
      // exact 64-bit keys of (s', index) over all slots
      auto slot = [&](int j) {
        const uint32_t* c = cw + 2 * kWave * min(j, kBSlots - 1);
        return j < min(cnt, kBSlots) ? KO::make(__uint_as_float(c[0]), (int)c[kWave]) : KO::pad();
      };
#pragma unroll
      for (int i = 0; i < 16; ++i) x[i] = slot(i);
      sort64_x16<KO>(x, g);
#pragma unroll 1
      for (int set = 1; 16 * set < kBSlots && __ballot(cnt > 16 * set) != 0; ++set) {
        K y[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) y[i] = slot(16 * set + i);
        sort64_x16<KO>(y, g);
        merge64_x16<KO>(x, y, g);
      }
      // x holds the best 64 by s', sorted; b is added (the scores stay
      // non-increasing, and ties that arise are put in order below)
#pragma unroll
      for (int i = 0; i < 16; ++i) x[i] = KO::make(KO::score(x[i]) + my_b, KO::index(x[i]));
    }
    // two entries whose scores are equal must stand in index order: the rare
    // row where some do not is sorted again
    bool disorder = false;
#pragma unroll
    for (int i = 1; i < 16; ++i) disorder |= KO::gt(x[i], x[i - 1]);
    {  // entry 16 (g + 1) of the row, held by the lane 16 above
      const uint32_t hi = (uint32_t)__shfl_down((int)(uint32_t)(x[0] >> 32), 16, kWave);
      const uint32_t lo = (uint32_t)__shfl_down((int)(uint32_t)x[0], 16, kWave);
      disorder |= g < 3 && KO::gt(((uint64_t)hi << 32) | lo, x[15]);
    }
    if (__ballot(disorder) != 0) sort64_x16<KO>(x, g);
    if (row_ok) {
      const size_t rw = bh * Q + my_row;
      // a lane's 16 entries are 64 contiguous bytes of its row
      const bool vec = k == kMaxK && ((reinterpret_cast<uintptr_t>(top_idx) |
                                       reinterpret_cast<uintptr_t>(top_score)) & 15) == 0;
      if (n_chunks == 1 && vec) {
        int4* ip = reinterpret_cast<int4*>(top_idx + rw * kMaxK + 16 * g);
#pragma unroll
        for (int u = 0; u < 4; ++u)
          ip[u] = int4{out_index<KO>(x[4 * u]), out_index<KO>(x[4 * u + 1]),
                       out_index<KO>(x[4 * u + 2]), out_index<KO>(x[4 * u + 3])};
        if (top_score) {
          float4* sp = reinterpret_cast<float4*>(top_score + rw * kMaxK + 16 * g);
#pragma unroll
          for (int u = 0; u < 4; ++u)
            sp[u] = float4{KO::score(x[4 * u]), KO::score(x[4 * u + 1]), KO::score(x[4 * u + 2]),
                           KO::score(x[4 * u + 3])};
        }
      } else if (n_chunks == 1) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int e = 16 * g + i;
          if (e < k) {
            top_idx[rw * k + e] = out_index<KO>(x[i]);
            if (top_score) top_score[rw * k + e] = KO::score(x[i]);
          }
        }
      } else {
#pragma unroll
        for (int i = 0; i < 16; ++i) part[(rw * n_chunks + ch) * kMaxK + 16 * g + i] = x[i];
      }
    }
    return;
  }

  // ---- fallback: online selection over the chunk, in two halves of 8 rows,
  // scores formed whole (accumulators starting at b)
  sc.init = my_b;
  wave_lds_sync();
  float* stage = reinterpret_cast<float*>(wl);  // [16][64], key column swizzled
  K* lists = reinterpret_cast<K*>(wl + kMR * kTile * 4);
  constexpr int kHalf = kMR / 2;
  for (int half = 0; half < 2; ++half) {
    RowLists<KO, kHalf> top;
    top.init(lists, lists + kHalf * kList);
    sc.for_tiles(hbase, kbeg, kend, kTile, qi, g, [&](int t0, f32x4_t* acc) {
#pragma unroll
      for (int sub = 0; sub < 4; ++sub) {
        const f32x4_t sv = acc[sub];
        *reinterpret_cast<f32x4_t*>(&stage[qi * kTile + ((16 * sub + 4 * g) ^ (qi << 2))]) = sv;
      }
      wave_lds_sync();
      const bool need_mask = t0 + kTile > kmin;
      for (int rr = 0; rr < kHalf; ++rr) {
        const int r = kHalf * half + rr;
        float sv = stage[r * kTile + (lane ^ (r << 2))];
        const int j = t0 + lane;
        if (need_mask && j >= __builtin_amdgcn_readlane(my_lim, r)) sv = -INFINITY;
        top.offer(rr, sv, j);
      }
      wave_lds_sync();
    });
    for (int rr = 0; rr < kHalf; ++rr) {
      top.finish(rr);
      const int i = row0 + kHalf * half + rr;
      if (i >= Q) continue;
      const K e = top.entry(rr);
      const size_t rw = bh * Q + i;
      if (n_chunks == 1) {
        if (lane < k) {
          top_idx[rw * k + lane] = out_index<KO>(e);
          if (top_score) top_score[rw * k + lane] = KO::score(e);
        }
      } else {
        part[(rw * n_chunks + ch) * kMaxK + lane] = e;
      }
    }
    wave_lds_sync();
  }
}

// ---------------------------------------------------------------- sketch scoring, MFMA, one pass

// Long rows (a batch of decode queries over a long cache) read each code once.
// A wave scores its 16 query rows against one key chunk on the MFMA (the
// layout of MfmaScorer, the mean term b folded into the accumulator) and
// keeps a running top-64 per row: a sorted 64-entry list and a 64-slot
// buffer of unsorted candidates, both in LDS.  A score is a candidate when it
// beats the row's threshold; a buffer that would overflow is sorted and
// merged into the list, which raises the threshold to the list's 64th score.
// Tiles are visited in increasing key order and buffers are flushed only
// between tiles, so a later key that merely ties the threshold ranks below
// every list entry: the strict test loses nothing.
//
// The threshold starts at a gate read off a sample of the chunk (8 tiles
// spread over it): the least, over the row's four lanes, of each lane's
// second-best sampled score, so that at least 8 sampled keys reach it.  The
// gate only bounds which keys are kept: a row whose list ends with 64
// entries above it holds the exact top-64 of the chunk.  A row that kept
// fewer (the gate was above its 64th score) still holds every key of the
// chunk above the gate.  With one chunk per row the wave scans such rows
// again without a gate.  With several, it records the gate in `gates` (-inf
// for rows that need none) and merge_kernel checks that the row's merged
// k-th score lies above every recorded gate, which makes the merged list
// exact.  Rows that fail the check are flagged; a second launch of this
// kernel with `only` = the flags rescans their chunks without a gate (its
// waves without a flagged row exit at once) and a second merge of just those
// rows follows.  A chunk's gate sits near its 200th-best key while the
// merged k-th score sits near each chunk's (64 / chunks)-th best, so rows
// fail only when several of their best keys fall in one chunk's sample (the
// queries of a sequence can share a few dominant keys).
//
// grid: 8 * ceil(ceil(units / kScanWaves) / 8) work-groups (XCD-ordered, as
// for xcd_logical_block), units = n_bh * wave_rows * n_chunks, one unit
// (head, 16-row block, chunk) per wave, chunks fastest.
using saki::kScanWaves;
constexpr int kScanBuf = 64;            // candidate slots per row
constexpr int kScanSample = 8;          // sampled tiles per chunk
constexpr int kScanGateKeys = 16 * kTile;  // rows with fewer keys in the chunk start ungated

template <int RK, int ST>
__global__ __launch_bounds__(kScanWaves * kWave) void score_scan_kernel(
    const uint8_t* __restrict__ index, int n_tiles, int N_valid, int Q,
    const int* __restrict__ q_pos, const float* __restrict__ q, const float* __restrict__ Bq,
    const float* __restrict__ mu, int H_q, int H_kv, int gq, int n_bh, int wave_rows, int chunk,
    int n_chunks, int k, int* __restrict__ top_idx, float* __restrict__ top_score,
    uint64_t* __restrict__ part, float* __restrict__ gates, const int* __restrict__ only) {
  constexpr int D = saki::kHeadDim;
  using KO = KeysF32;
  using K = KO::K;
  using Scorer = MfmaScorer<RK, ST>;
  __shared__ K list_mem[kScanWaves][kMR * kList];
  __shared__ K buf_mem[kScanWaves][kMR * kScanBuf];  // first the sketch staging [16][RK] floats
  static_assert(kMR * RK * sizeof(float) <= kMR * kScanBuf * sizeof(K), "sketch staging fits");
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = lane_id();
  const long long units = (long long)n_bh * wave_rows * n_chunks;
  const long long lb = xcd_logical_block((units + kScanWaves - 1) / kScanWaves);
  if (lb < 0) return;
  const long long unit = lb * kScanWaves + wave;
  if (unit >= units) return;
  const int ch = (int)(unit % n_chunks);
  const int wr = (int)((unit / n_chunks) % wave_rows);
  const size_t bh = (size_t)(unit / ((long long)n_chunks * wave_rows));
  const int h = (int)(bh % H_q);
  const int qi = lane % 16, g = lane / 16;
  const int row0 = wr * kMR;
  const int my_row = row0 + qi;
  const bool row_ok = my_row < Q;
  // with `only`, the rows to redo (a wave with none has nothing to do)
  const bool want = row_ok && (!only || only[bh * Q + my_row] != 0);
  if (only && __ballot(want) == 0) return;
  const int my_lim = row_limit(my_row, Q, N_valid, q_pos);
  const int kmax = wave_max_i(my_lim);
  const int kmin = wave_min_i(row_ok ? my_lim : INT_MAX);
  const int kbeg = ch * chunk;
  const int kend = min(kbeg + chunk, kmax);
  K* list = list_mem[wave];
  K* buf = buf_mem[wave];

  const size_t code_set = (bh / H_q) * (H_q / gq) + h / gq;
  const uint8_t* hbase = index + code_set * n_tiles * Scorer::TB;
  // the gate's sample: every stride-th tile of the chunk, at most kScanSample;
  // the first kSA of them are requested before the query sketch is formed
  const int n_row = row_ok ? max(0, min(my_lim, kend) - kbeg) : 0;
  const bool gated = !only && wave_max_i(n_row) >= kScanGateKeys;
  const int stride = max(1, (kend - kbeg) / (kTile * kScanSample)) * kTile;
  const int n_samp = gated ? min(kScanSample, (kend - kbeg + stride - 1) / stride) : 0;
  constexpr int kSA = Scorer::NL == 1 ? 4 : Scorer::kPrefetch ? 2 : 1;
  Scorer sc;
  typename Scorer::Raw sraw[kSA];
  auto sample_at = [&](int i) { return hbase + (size_t)((kbeg + i * stride) / kTile) * Scorer::TB; };
#pragma unroll
  for (int u = 0; u < kSA; ++u)
    if (u < n_samp) sc.load(sample_at(u), qi, g, sraw[u]);

  sc.init = mfma_query_sketch<RK, ST>(q + (bh * Q + (row_ok ? my_row : row0)) * D, row_ok,
                                      Bq + (size_t)h * D * RK, mu + (size_t)(h / (H_q / H_kv)) * D,
                                      reinterpret_cast<float*>(buf), qi, g, sc);
#pragma unroll 1
  for (int r = 0; r < kMR; ++r) list[r * kList + lane] = KO::pad();

  // ---- the gate
  float tau = -INFINITY;
  if (gated) {
    float m1 = -INFINITY, m2 = -INFINITY;
    for (int i0 = 0; i0 < n_samp; i0 += kSA) {
#pragma unroll
      for (int u = 0; u < kSA; ++u) {
        const int i = i0 + u;
        if (i >= n_samp) break;
        f32x4_t acc[4];
        sc.mma(sraw[u], acc);
        if (i + kSA < n_samp) sc.load(sample_at(i + kSA), qi, g, sraw[u]);
        const int t0 = kbeg + i * stride;
#pragma unroll
        for (int sub = 0; sub < 4; ++sub)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const float x = t0 + 16 * sub + 4 * g + v < my_lim ? acc[sub][v] : -INFINITY;
            m2 = fmaxf(m2, fminf(m1, x));
            m1 = fmaxf(m1, x);
          }
      }
    }
    // the least of the four lanes' second-best sampled scores: at least 8
    // sampled keys reach it
    float m = m2;
    m = fminf(m, xor_shfl_f32(m, 16));
    m = fminf(m, xor_shfl_f32(m, 32));
    if (n_row >= kScanGateKeys) tau = m;
  }

  // ---- the scan
  float thr = want ? tau : INFINITY;  // row qi's threshold (the same in its four lanes)
  int base = 0;                       // row qi's buffered candidates
  auto flush = [&](int r) {
    wave_lds_sync();
    const int c = __builtin_amdgcn_readlane(base, r);  // lane r: row r, lane group 0
    K b = lane < c ? buf[r * kScanBuf + lane] : KO::pad();
    wave_sort<KO>(b);
    K a = list[r * kList + lane];
    wave_merge<KO>(a, b);
    list[r * kList + lane] = a;
    const float t = KO::score(KO::readlane(a, kWave - 1));
    if (qi == r) {
      thr = fmaxf(thr, t);
      base = 0;
    }
    wave_lds_sync();
  };
  auto scan = [&]() {
    sc.for_tiles_deep(hbase, kbeg, kend, qi, g, [&](int t0, f32x4_t* acc) {
      uint32_t take = 0;
#pragma unroll
      for (int sub = 0; sub < 4; ++sub)
#pragma unroll
        for (int v = 0; v < 4; ++v) take |= (acc[sub][v] > thr ? 1u : 0u) << (4 * sub + v);
      if (t0 + kTile > kmin) {  // a tile crossing some row's limit
#pragma unroll
        for (int sub = 0; sub < 4; ++sub)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (t0 + 16 * sub + 4 * g + v >= my_lim) take &= ~(1u << (4 * sub + v));
      }
      if (__ballot(take != 0) == 0) return;
      // the four lanes of a row append at offsets from a prefix of their counts
      int c = __popc(take);
      int c1 = (int)xor_shfl_u32((uint32_t)c, 16);   // lane group g ^ 1
      int c2 = (int)xor_shfl_u32((uint32_t)c, 32);   // g ^ 2
      int c3 = (int)xor_shfl_u32((uint32_t)c1, 32);  // g ^ 3
      uint64_t full = __ballot(base + c + c1 + c2 + c3 > kScanBuf) & 0xffffull;
      if (full) {
        do {
          flush(__builtin_ctzll(full));
          full &= full - 1;
        } while (full);
#pragma unroll
        for (int sub = 0; sub < 4; ++sub)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (!(acc[sub][v] > thr)) take &= ~(1u << (4 * sub + v));
        c = __popc(take);
        c1 = (int)xor_shfl_u32((uint32_t)c, 16);
        c2 = (int)xor_shfl_u32((uint32_t)c, 32);
        c3 = (int)xor_shfl_u32((uint32_t)c1, 32);
      }
      int pos = base + (g == 1 ? c1 : g == 2 ? c2 + c3 : g == 3 ? c1 + c2 + c3 : 0);
      base += c + c1 + c2 + c3;
      // a lane rarely holds more than one or two candidates of a tile: take
      // them one per round, lowest element first, each picked out of the 16
      // scores by the bits of its element number
      while (__ballot(take != 0)) {
        const int e = __builtin_ctz(take | 0x10000u);
        // bit masks of e's bits: (m & x) | (~m & y) picks x where the bit is set
        const uint32_t m0 = 0u - (uint32_t)(e & 1), m1 = 0u - (uint32_t)((e >> 1) & 1);
        const uint32_t m2 = 0u - (uint32_t)((e >> 2) & 1), m3 = 0u - (uint32_t)((e >> 3) & 1);
        auto pick = [](uint32_t m, uint32_t x, uint32_t y) { return (m & x) | (~m & y); };
        uint32_t s8[8], s4[4], s2[2];
#pragma unroll
        for (int m = 0; m < 8; ++m)
          s8[m] = pick(m0, __float_as_uint(acc[m >> 1][(2 * m + 1) & 3]), __float_as_uint(acc[m >> 1][(2 * m) & 3]));
#pragma unroll
        for (int m = 0; m < 4; ++m) s4[m] = pick(m1, s8[2 * m + 1], s8[2 * m]);
#pragma unroll
        for (int m = 0; m < 2; ++m) s2[m] = pick(m2, s4[2 * m + 1], s4[2 * m]);
        const float sv = __uint_as_float(pick(m3, s2[1], s2[0]));
        if (take) {
          buf[qi * kScanBuf + pos] = KO::make(sv, t0 + 16 * (e >> 2) + 4 * g + (e & 3));
          ++pos;
          take &= take - 1;
        }
      }
    });
    uint64_t left = __ballot(base > 0) & 0xffffull;
    while (left) {
      flush(__builtin_ctzll(left));
      left &= left - 1;
    }
  };
  scan();
  // rows whose gate kept fewer than 64 keys of the chunk
  wave_lds_sync();
  const bool short_row = tau > -INFINITY && KO::index(list[qi * kList + kList - 1]) == kPadIdx;
  if (n_chunks > 1) {
    if (g == 0 && want) gates[(bh * Q + my_row) * n_chunks + ch] = short_row ? tau : -INFINITY;
  } else if (__ballot(short_row) != 0) {  // one chunk: again, ungated; the other rows are done
    for (uint64_t m = __ballot(short_row) & 0xffffull; m; m &= m - 1)
      list[__builtin_ctzll(m) * kList + lane] = KO::pad();
    thr = short_row ? -INFINITY : INFINITY;
    wave_lds_sync();
    scan();
    wave_lds_sync();
  }

  for (int r = 0; r < kMR; ++r) {
    const int i = row0 + r;
    if (i >= Q) break;
    if (!__builtin_amdgcn_readlane((int)want, r)) continue;
    const K e = list[r * kList + lane];
    if (n_chunks == 1) {
      if (lane < k) {
        const size_t o = (bh * Q + i) * k + lane;
        top_idx[o] = out_index<KO>(e);
        if (top_score) top_score[o] = KO::score(e);
      }
    } else {
      part[((bh * Q + i) * n_chunks + ch) * kMaxK + lane] = e;
    }
  }
}

// ---------------------------------------------------------------- exact scores + recall

// Writes the exact top-k of a finished row, or its partial list.
template <class KO>
__device__ __forceinline__ void exact_row_out(typename KO::K e, size_t row, int ch, int n_chunks,
                                              int k, const int* approx, int* hits,
                                              int* exact_idx, typename KO::K* part) {
  const int lane = lane_id();
  if (n_chunks == 1) {
    const int ej = out_index<KO>(e);
    if (exact_idx && lane < k) exact_idx[row * k + lane] = ej;
    const int hsum = row_hits(ej, approx, row, k);
    if (lane == 0) hits[row] = hsum;
  } else {
    part[(row * n_chunks + ch) * kMaxK + lane] = e;
  }
}

// grid (row_blocks * n_chunks, B*H_q), block 64*waves.  Exact float64 scores
// with float64 FMAs, one key per lane, R rows per wave.
template <bool KBF, int R>
__global__ __launch_bounds__(256) void exact_stream_kernel(
    const void* __restrict__ keys, const float* __restrict__ q,
    const int* __restrict__ q_pos, int H_q, int H_kv, int N_cap, int N_valid, int Q,
    int row_blocks, int chunk, int n_chunks, int k, const int* __restrict__ approx,
    int* __restrict__ hits, int* __restrict__ exact_idx, KeyF64* __restrict__ part) {
  constexpr int D = saki::kHeadDim;
  using KO = KeysF64;
  __shared__ double qsh[kStreamWaves][R][D];
  __shared__ KeyF64 lmem[kStreamWaves][R][kList];
  __shared__ KeyF64 bmem[kStreamWaves][R][kList];
  const int wave = threadIdx.x / kWave, lane = lane_id();
  const int waves = blockDim.x / kWave;
  const int rb = blockIdx.x % row_blocks, ch = blockIdx.x / row_blocks;
  const size_t bh = blockIdx.y;
  const int b = (int)(bh / H_q), h = (int)(bh % H_q);
  const int gkv = h / (H_q / H_kv);
  const int row0 = (rb * waves + wave) * R;
  if (row0 >= Q) return;
  int lim[R];
  int kmax = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    lim[r] = row_limit(row0 + r, Q, N_valid, q_pos);
    kmax = lim[r] > kmax ? lim[r] : kmax;
  }
  for (int i = lane; i < R * D; i += kWave) {
    const int r = i / D;
    qsh[wave][r][i % D] = (row0 + r < Q) ? (double)q[(bh * Q + row0 + r) * D + (i % D)] : 0.0;
  }
  RowLists<KO, R> top;
  top.init(&lmem[wave][0][0], &bmem[wave][0][0]);
  const size_t kbase = ((size_t)b * H_kv + gkv) * N_cap;
  const int kbeg = ch * chunk;
  const int kend = min(kbeg + chunk, kmax);
  for (int t0 = kbeg; t0 < kend; t0 += kTile) {
    const int j = t0 + lane;
    const bool inb = j < N_valid;
    double acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.0;
#pragma unroll 2
    for (int c0 = 0; c0 < D; c0 += 8) {
      double kv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) kv[e] = inb ? (double)load_key_elem<KBF>(keys, (kbase + j) * D + c0 + e) : 0.0;
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[r] = fma(qsh[wave][r][c0 + e], kv[e], acc[r]);
    }
#pragma unroll
    for (int r = 0; r < R; ++r) top.offer(r, j < lim[r] ? acc[r] : -(double)INFINITY, j);
  }
  for (int r = 0; r < R; ++r) {
    top.finish(r);
    const int i = row0 + r;
    if (i >= Q) continue;
    exact_row_out<KO>(top.entry(r), bh * Q + i, ch, n_chunks, k, approx, hits, exact_idx, part);
  }
}

// Exact float64 scores on the f64 MFMA (16x16x4).  Lane group g feeds dims
// 32g .. 32g+31 of its key and query, one per k-step.  The f64 MFMA returns
// D[g + 4v][lane % 16] in register v.  grid (row_blocks * n_chunks, B*H_q) via
// xcd_grid, two waves of 16 rows per work-group.
template <bool KBF>
__global__ __launch_bounds__(128) void exact_mfma_kernel(
    const void* __restrict__ keys, const float* __restrict__ q,
    const int* __restrict__ q_pos, int H_q, int H_kv, int N_cap, int N_valid, int Q,
    int row_blocks, int chunk, int n_chunks, int k, const int* __restrict__ approx,
    int* __restrict__ hits, int* __restrict__ exact_idx, KeyF64* __restrict__ part, int n_bh,
    const int* __restrict__ redo) {
  constexpr int D = saki::kHeadDim;
  using KO = KeysF64;
  // staged scores [row][key], key column swizzled by the row index
  __shared__ double stage[kMfmaWaves][kMR][kTile];
  __shared__ KeyF64 lmem[kMfmaWaves][kMR][kList];
  __shared__ KeyF64 bmem[kMfmaWaves][kMR][kList];
  const int wave = threadIdx.x / kWave, lane = lane_id();
  const int waves = blockDim.x / kWave;
  const long long lb = xcd_logical_block((long long)row_blocks * n_chunks * n_bh);
  if (lb < 0) return;
  const int rb = (int)(lb % row_blocks), ch = (int)((lb / row_blocks) % n_chunks);
  const size_t bh = (size_t)(lb / ((long long)row_blocks * n_chunks));
  const int b = (int)(bh / H_q), h = (int)(bh % H_q);
  const int gkv = h / (H_q / H_kv);
  const int row0 = (rb * waves + wave) * kMR;
  if (row0 >= Q) return;
  // as the fallback of exact_bf16_kernel: only the waves it flagged
  if (redo && redo[lb * kMfmaWaves + wave] == 0) return;
  const int qi = lane % 16, g = lane / 16;
  const int my_row = row0 + qi;
  const bool row_ok = my_row < Q;
  const int my_lim = row_limit(my_row, Q, N_valid, q_pos);
  const int kmax = wave_max_i(my_lim);
  const int kmin = wave_min_i(row_ok ? my_lim : INT_MAX);
  double qreg[32];
  {
    const float* qr = q + (bh * Q + (row_ok ? my_row : row0)) * D + 32 * g;
#pragma unroll
    for (int s4 = 0; s4 < 8; ++s4) {
      const float4 v = *reinterpret_cast<const float4*>(qr + 4 * s4);
      qreg[4 * s4 + 0] = row_ok ? (double)v.x : 0.0;
      qreg[4 * s4 + 1] = row_ok ? (double)v.y : 0.0;
      qreg[4 * s4 + 2] = row_ok ? (double)v.z : 0.0;
      qreg[4 * s4 + 3] = row_ok ? (double)v.w : 0.0;
    }
  }
  RowLists<KO, kMR> top;
  top.init(&lmem[wave][0][0], &bmem[wave][0][0]);
  const size_t kbase = ((size_t)b * H_kv + gkv) * N_cap;
  const int kbeg = ch * chunk;
  const int kend = min(kbeg + chunk, kmax);
  for (int t0 = kbeg; t0 < kend; t0 += kTile) {
#pragma unroll
    for (int sub = 0; sub < 4; ++sub) {
      const int j = t0 + 16 * sub + qi;
      const bool inb = j < N_valid;
      float kf[32];
      if constexpr (KBF) {
        const uint16_t* kr = reinterpret_cast<const uint16_t*>(keys) + (kbase + (inb ? j : 0)) * D + 32 * g;
#pragma unroll
        for (int s8 = 0; s8 < 4; ++s8) {
          const uint4 v = *reinterpret_cast<const uint4*>(kr + 8 * s8);
          unpack_piece<true>(v, kf + 8 * s8);
        }
      } else {
        const float* kr = reinterpret_cast<const float*>(keys) + (kbase + (inb ? j : 0)) * D + 32 * g;
#pragma unroll
        for (int s4 = 0; s4 < 8; ++s4) {
          const float4 v = *reinterpret_cast<const float4*>(kr + 4 * s4);
          kf[4 * s4 + 0] = v.x;
          kf[4 * s4 + 1] = v.y;
          kf[4 * s4 + 2] = v.z;
          kf[4 * s4 + 3] = v.w;
        }
      }
      f64x4_t acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
      for (int s = 0; s < 32; ++s)
        acc = __builtin_amdgcn_mfma_f64_16x16x4f64(inb ? (double)kf[s] : 0.0, qreg[s], acc, 0, 0, 0);
#pragma unroll
      for (int v = 0; v < 4; ++v) stage[wave][qi][(16 * sub + g + 4 * v) ^ qi] = acc[v];
    }
    wave_lds_sync();
    const bool need_mask = t0 + kTile > kmin;
    for (int r = 0; r < kMR; ++r) {
      double sv = stage[wave][r][lane ^ r];
      const int j = t0 + lane;
      if (need_mask && j >= __builtin_amdgcn_readlane(my_lim, r)) sv = -(double)INFINITY;
      top.offer(r, sv, j);
    }
    wave_lds_sync();
  }
  for (int r = 0; r < kMR; ++r) {
    top.finish(r);
    const int i = row0 + r;
    if (i >= Q) continue;
    exact_row_out<KO>(top.entry(r), bh * Q + i, ch, n_chunks, k, approx, hits, exact_idx, part);
  }
}

// ---------------------------------------------------------------- exact scores, bound-and-rescore

// Keys rounded to bf16 in the MFMA tile layout of the codes (16 pieces of 8
// dims per key), and an upper bound of every key's Euclidean norm (rows of
// n_tiles * 64 per (b, g), so that aligned groups of four can be loaded).
// grid (n_tiles(N_valid), B*H_kv), block 256.
template <bool KBF>
__global__ __launch_bounds__(256) void keys_hi_kernel(const void* __restrict__ keys, int N_cap,
                                                      int N_valid, int n_tiles,
                                                      uint8_t* __restrict__ khi,
                                                      uint8_t* __restrict__ klo,
                                                      float* __restrict__ knorm) {
  constexpr int D = saki::kHeadDim;
  constexpr int NP = D / 8;
  __shared__ float part[4][kTile];
  const int tile = blockIdx.x;
  const size_t bg = blockIdx.y;
  const int t = threadIdx.x % kTile, pg = threadIdx.x / kTile;
  const int n = tile * kTile + t;
  const bool ok = n < N_valid;
  const size_t toff = (bg * n_tiles + tile) * (size_t)kTile * D * 2;
  float ss = 0.f;
  for (int p = pg; p < NP; p += 4) {
    float f[8], hi[8], lo[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      f[e] = ok ? load_key_elem<KBF>(keys, (bg * N_cap + n) * D + 8 * p + e) : 0.f;
      ss = fmaf(f[e], f[e], ss);
      hi[e] = bf16_round(f[e]);
      lo[e] = bf16_round(f[e] - hi[e]);  // exact difference, then rounded
    }
    const size_t o = toff + (size_t)p * kTile * 16 + (size_t)t * 16;
    *reinterpret_cast<uint4*>(khi + o) = pack_bf16x8(hi);
    *reinterpret_cast<uint4*>(klo + o) = pack_bf16x8(lo);
  }
  part[pg][t] = ss;
  __syncthreads();
  if (pg == 0)  // one row of n_tiles * 64 bounds per (b, g); 0 past N_valid
    knorm[bg * n_tiles * kTile + n] =
        ok ? sqrtf(part[0][t] + part[1][t] + part[2][t] + part[3][t]) * (1.f + 1e-5f) : 0.f;
}

// Exact top-64 and recall hits by bound-and-rescore.  With x = x_h + x_l + x_r
// (x_h = bf16(x), x_l = bf16(x - x_h)), the three bf16 MFMA products
// a3 = q_h.k_h + q_h.k_l + q_l.k_h miss q.k by the dropped terms (at most about
// 3 * 2^-16 sum|q_i k_i|) plus float32 accumulation (at most 384 * 2^-24 of the
// same sum), so |a3 - q.k| <= E = kExactEps3 * ||q|| ||k|| with 40% margin.
// Three passes run on these intervals: moments of the
// single product q_h.k_h (only a prediction), a histogram of the lower bounds
// a3 - E, and a gate on the upper bounds a3 + E at the bin where the
// lower-bound count reaches 64: every key whose exact score can reach the 64th
// exact score passes it.  Gated keys are rescored in float64 (float32 inputs,
// so every product is exact) and sorted.  A wave whose rows miss the
// prediction or gate more than 128 keys is flagged and redone by
// exact_mfma_kernel.  grid/block as exact_mfma_kernel.
constexpr float kExactEps3 = 1e-4f;

template <bool KBF>
__global__ __launch_bounds__(128) void exact_bf16_kernel(
    const void* __restrict__ keys, const uint8_t* __restrict__ khi,
    const uint8_t* __restrict__ klo, const float* __restrict__ knorm, const float* __restrict__ q,
    const int* __restrict__ q_pos, int H_q, int H_kv, int N_cap, int N_valid, int Q,
    int n_tiles_hi, int n_bh, int row_blocks, int chunk, int n_chunks, int k,
    const int* __restrict__ approx, int* __restrict__ hits, int* __restrict__ exact_idx,
    KeyF64* __restrict__ part, const int* __restrict__ only, int* __restrict__ redo) {
  constexpr int D = saki::kHeadDim;
  constexpr size_t TB = (size_t)kTile * D * 2;
  using KO = KeysF64;
  __shared__ int cand_mem[kMfmaWaves][kMR * kCandRow];
  __shared__ int hist_mem[kMfmaWaves][kMR * kHistRow];
  __shared__ float qrow_mem[kMfmaWaves][kMR * D];
  __shared__ int ccount[kMfmaWaves][kMR];
  const int wave = threadIdx.x / kWave, lane = lane_id();
  const int waves = blockDim.x / kWave;
  const long long lb = xcd_logical_block((long long)row_blocks * n_chunks * n_bh);
  if (lb < 0) return;
  const int rb = (int)(lb % row_blocks), ch = (int)((lb / row_blocks) % n_chunks);
  const size_t bh = (size_t)(lb / ((long long)row_blocks * n_chunks));
  const int b = (int)(bh / H_q), h = (int)(bh % H_q);
  const int gkv = h / (H_q / H_kv);
  const size_t bg = (size_t)b * H_kv + gkv;
  const int row0 = (rb * waves + wave) * kMR;
  if (row0 >= Q) return;
  // as the second tier after exact_gate_kernel: only the waves it flagged
  if (only && only[lb * kMfmaWaves + wave] == 0) {
    if (lane == 0) redo[lb * kMfmaWaves + wave] = 0;
    return;
  }
  const int qi = lane % 16, g = lane / 16;
  const int my_row = row0 + qi;
  const bool row_ok = my_row < Q;
  const int my_lim = row_limit(my_row, Q, N_valid, q_pos);
  const int kmax = wave_max_i(my_lim);
  const int kmin = wave_min_i(row_ok ? my_lim : INT_MAX);
  const int kbeg = ch * chunk;
  const int kend = min(kbeg + chunk, kmax);
  int* cand = cand_mem[wave];
  int* hist = hist_mem[wave];
  float* qrows = qrow_mem[wave];
  const size_t hoff = bg * n_tiles_hi * TB;
  const float* kn = knorm + bg * n_tiles_hi * kTile;

  // query: bf16 hi/lo operands (dims 32kk + 8g .. +7), float32 copy in LDS,
  // norm bound
  bf16x8_t qh[4], ql[4];
  float qn;
  {
    const float* qr = q + (bh * Q + (row_ok ? my_row : row0)) * D;
    float ss = 0.f;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      float fh[8], fl[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float f = row_ok ? qr[32 * kk + 8 * g + e] : 0.f;
        ss = fmaf(f, f, ss);
        qrows[qi * D + 32 * kk + 8 * g + e] = f;
        fh[e] = bf16_round(f);
        fl[e] = bf16_round(f - fh[e]);
      }
      qh[kk] = as_bf16x8(pack_bf16x8(fh));
      ql[kk] = as_bf16x8(pack_bf16x8(fl));
    }
    qn = sqrtf(sum_lane_groups(ss)) * (1.f + 1e-5f);
  }
  const float eq = kExactEps3 * qn;
  wave_lds_sync();

  // THREE: a3 (three products) and its error radius; otherwise q_h.k_h only.
  auto tile = [&](int t0, f32x4_t acc[4], float e[4][4], auto three) {
    const size_t to = hoff + (size_t)(t0 / kTile) * TB;
#pragma unroll
    for (int sub = 0; sub < 4; ++sub) {
      const int key = 16 * sub + qi;
      f32x4_t a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const size_t o = to + (size_t)(4 * kk + g) * kTile * 16 + (size_t)key * 16;
        const bf16x8_t kh = as_bf16x8(*reinterpret_cast<const uint4*>(khi + o));
        a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kh, qh[kk], a, 0, 0, 0);
        if constexpr (decltype(three)::value) {
          const bf16x8_t kl = as_bf16x8(*reinterpret_cast<const uint4*>(klo + o));
          a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kl, qh[kk], a, 0, 0, 0);
          a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kh, ql[kk], a, 0, 0, 0);
        }
      }
      acc[sub] = a;
      if constexpr (decltype(three)::value) {
        // radii of keys t0 + 16 sub + 4g .. +3 (keys past N_valid are masked)
        const int kb = t0 + 16 * sub + 4 * g;
#pragma unroll
        for (int v = 0; v < 4; ++v) e[sub][v] = (kb + v < N_valid) ? eq * kn[kb + v] : 0.f;
      }
    }
  };
  using One = std::integral_constant<bool, false>;
  using Three = std::integral_constant<bool, true>;

  // ---- pass 1: moments of the approximate scores
  float sum = 0.f, sumsq = 0.f;
  for (int t0 = kbeg; t0 < kend; t0 += kTile) {
    f32x4_t acc[4];
    float e[4][4];
    tile(t0, acc, e, One{});
    const bool need_mask = t0 + kTile > kmin;
#pragma unroll
    for (int sub = 0; sub < 4; ++sub)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        float x = acc[sub][v];
        if (need_mask && t0 + 16 * sub + 4 * g + v >= my_lim) x = 0.f;
        sum += x;
        sumsq = fmaf(x, x, sumsq);
      }
  }
  sum = sum_lane_groups(sum);
  sumsq = sum_lane_groups(sumsq);
  const int n_row = row_ok ? max(0, min(my_lim, kend) - kbeg) : 0;
  int mode = kModeAll;
  float inv_w = 0.f, off = 0.f;
  if (n_row > kCollect) {
    const float mean = sum / (float)n_row;
    const float sd = sqrtf(fmaxf(sumsq / (float)n_row - mean * mean, 0.f));
    if (sd > 0.f && isfinite(sd) && isfinite(mean)) {
      const float t_hat = mean + sd * normal_upper_quantile((float)kList / (float)n_row);
      const float lo = t_hat - 2.f * sd;
      inv_w = (float)(kBins - 2) / (3.f * sd);
      off = 1.f - lo * inv_w;
      mode = kModeHist;
    } else {
      mode = kModeFallback;
    }
  }

  // ---- pass 2: histogram of the lower bounds
  float gate = -INFINITY;
  if (__ballot(mode == kModeHist) != 0) {
    for (int i = lane; i < kMR * kHistRow; i += kWave) hist[i] = 0;
    wave_lds_sync();
    for (int t0 = kbeg; t0 < kend; t0 += kTile) {
      f32x4_t acc[4];
      float e[4][4];
      tile(t0, acc, e, Three{});
#pragma unroll
      for (int sub = 0; sub < 4; ++sub)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float x = fmaf(acc[sub][v] - e[sub][v], inv_w, off);
          if (mode == kModeHist && x >= 1.f && t0 + 16 * sub + 4 * g + v < my_lim)
            atomicAdd(&hist[qi * kHistRow + min((int)x, kBins - 1)], 1);
        }
    }
    wave_lds_sync();
    for (int r = 0; r < kMR; ++r) {
      if (__builtin_amdgcn_readlane(mode, r) != kModeHist) continue;
      int x = hist[r * kHistRow + (kBins - 1 - lane)];
      if (lane == kBins - 1) x = 0;
#pragma unroll
      for (int d = 1; d < kWave; d <<= 1) {
        const int t = __shfl_up(x, d, kWave);
        if (lane >= d) x += t;
      }
      const uint64_t reach = __ballot(x >= kList);
      const int new_mode = reach == 0 ? (int)kModeFallback : (int)kModeHist;
      const float bstar = reach == 0 ? 0.f : (float)(kBins - 1 - __builtin_ctzll(reach));
      if (qi == r) {
        mode = new_mode;
        gate = bstar;
      }
    }
  }

  // ---- pass 3: collect the keys whose upper bound reaches the gate
  bool fallback = __ballot(mode == kModeFallback) != 0;
  if (!fallback) {
    if (lane < kMR) ccount[wave][lane] = 0;
    wave_lds_sync();
    for (int t0 = kbeg; t0 < kend; t0 += kTile) {
      f32x4_t acc[4];
      float e[4][4];
      tile(t0, acc, e, Three{});
#pragma unroll
      for (int sub = 0; sub < 4; ++sub)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int key = t0 + 16 * sub + 4 * g + v;
          const bool take = key < my_lim &&
                            (mode == kModeAll || fmaf(acc[sub][v] + e[sub][v], inv_w, off) >= gate);
          if (take) {
            const int pos = atomicAdd(&ccount[wave][qi], 1);
            if (pos < kCollect) cand[qi * kCandRow + pos] = key;
          }
        }
    }
    wave_lds_sync();
    fallback = __ballot(lane < kMR && ccount[wave][lane < kMR ? lane : 0] > kCollect) != 0;
  }
  if (lane == 0) redo[lb * kMfmaWaves + wave] = fallback ? 1 : 0;
  if (fallback) return;

  // ---- rescoring in float64 and the exact top-64 of each row
  const size_t kbase = bg * N_cap;
  for (int r = 0; r < kMR; ++r) {
    const int i = row0 + r;
    if (i >= Q) break;
    const int c = ccount[wave][r];
    KeyF64 best = KO::pad();
    for (int base = 0; base < c; base += kWave) {
      KeyF64 x = KO::pad();
      if (base + lane < c) {
        const int j = cand[r * kCandRow + base + lane];
        double acc = 0.0;
        if constexpr (KBF) {
          const uint16_t* kr = reinterpret_cast<const uint16_t*>(keys) + (kbase + j) * D;
#pragma unroll 4
          for (int d8 = 0; d8 < D; d8 += 8) {
            float f[8];
            unpack_piece<true>(*reinterpret_cast<const uint4*>(kr + d8), f);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc = fma((double)qrows[r * D + d8 + e], (double)f[e], acc);
          }
        } else {
          const float* kr = reinterpret_cast<const float*>(keys) + (kbase + j) * D;
#pragma unroll 4
          for (int d4 = 0; d4 < D; d4 += 4) {
            const float4 f = *reinterpret_cast<const float4*>(kr + d4);
            acc = fma((double)qrows[r * D + d4 + 0], (double)f.x, acc);
            acc = fma((double)qrows[r * D + d4 + 1], (double)f.y, acc);
            acc = fma((double)qrows[r * D + d4 + 2], (double)f.z, acc);
            acc = fma((double)qrows[r * D + d4 + 3], (double)f.w, acc);
          }
        }
        x = KO::make(acc, j);
      }
      wave_sort<KO>(x);
      if (base == 0) best = x;
      else wave_merge<KO>(best, x);
    }
    exact_row_out<KO>(best, bh * Q + i, ch, n_chunks, k, approx, hits, exact_idx, part);
  }
}

// ---------------------------------------------------------------- exact scores, gated by the candidate list

// The k-th best exact score among any k distinct visible keys is a lower
// bound of the row's exact k-th score, so the candidate list S_i itself gives
// every row a gate tau_i before the scan.  The gate is taken from float32 dot
// products, whose error is at most gamma_128 sum|q_e k_e| <= 7.7e-6 ||q|| ||k||.
constexpr float kTauEps = 1e-5f;

// Order-preserving 32-bit key of a float score whose low 7 bits carry a slot
// number (0..127); 0 is never produced for a finite score and marks a pad.
__device__ __forceinline__ uint32_t slot_key(float s, int slot) {
  return (ord_f32(s) & ~127u) | (uint32_t)slot;
}

__device__ __forceinline__ float wave_min_f32(float v) {
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) v = fminf(v, xor_shfl_f32(v, m));
  return v;
}
__device__ __forceinline__ float wave_max_f32(float v) {
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) v = fmaxf(v, xor_shfl_f32(v, m));
  return v;
}

// Float32 q.k of one key per lane (four partial sums); q in LDS.
template <bool KBF>
__device__ __forceinline__ float lane_dot_f32(const void* keys, size_t key_row, const float* qs) {
  constexpr int D = saki::kHeadDim;
  float s[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int d8 = 0; d8 < D; d8 += 8) {
    float f[8];
    if constexpr (KBF) {
      unpack_piece<true>(*reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(keys) +
                                                         key_row * D + d8), f);
    } else {
      const float4* kr = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(keys) +
                                                         key_row * D + d8);
      const float4 a = kr[0], b = kr[1];
      f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
      f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e & 3] = fmaf(qs[d8 + e], f[e], s[e & 3]);
  }
  return (s[0] + s[1]) + (s[2] + s[3]);
}

// Float64 q.k of one key per lane (float32 inputs: every product is exact).
template <bool KBF>
__device__ __forceinline__ double lane_dot_f64(const void* keys, size_t key_row, const float* qs) {
  constexpr int D = saki::kHeadDim;
  double acc = 0.0;
#pragma unroll 4
  for (int d8 = 0; d8 < D; d8 += 8) {
    float f[8];
    if constexpr (KBF) {
      unpack_piece<true>(*reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(keys) +
                                                         key_row * D + d8), f);
    } else {
      const float4* kr = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(keys) +
                                                         key_row * D + d8);
      const float4 a = kr[0], b = kr[1];
      f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
      f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = fma((double)qs[d8 + e], (double)f[e], acc);
  }
  return acc;
}

// Whether j is in a row's candidate list, kept sorted descending in LDS
// (64 entries; unused slots hold values >= 2^31, which no index equals).
__device__ __forceinline__ bool in_sorted_desc(const uint32_t* a, int j) {
  if (j < 0) return false;
  const uint32_t x = (uint32_t)j;
  int lo = 0;
#pragma unroll
  for (int st = 32; st > 0; st >>= 1)
    if (a[lo + st - 1] > x) lo += st;
  return lo < kWave && a[lo] == x;
}

// Float64 q.k of one key per lane, q read from global memory.
template <bool KBF>
__device__ __forceinline__ double lane_dot_f64_g(const void* keys, size_t key_row,
                                                 const float* __restrict__ qr) {
  constexpr int D = saki::kHeadDim;
  double acc = 0.0;
#pragma unroll 2
  for (int d8 = 0; d8 < D; d8 += 8) {
    float f[8];
    if constexpr (KBF) {
      unpack_piece<true>(*reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(keys) +
                                                         key_row * D + d8), f);
    } else {
      const float4* kr = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(keys) +
                                                         key_row * D + d8);
      const float4 a = kr[0], b = kr[1];
      f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
      f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
    }
    const float4 qa = *reinterpret_cast<const float4*>(qr + d8);
    const float4 qb = *reinterpret_cast<const float4*>(qr + d8 + 4);
    const float qv[8] = {qa.x, qa.y, qa.z, qa.w, qb.x, qb.y, qb.z, qb.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = fma((double)qv[e], (double)f[e], acc);
  }
  return acc;
}

constexpr int kGateCap = 64;            // keys one wave collects per row
constexpr int kGateRow = kGateCap + 1;  // row stride; slot kGateCap absorbs overflow writes
constexpr int kBatch = 160;             // keys rescored per wave and batch
constexpr int kGateWaves = 4;           // waves per 16-row work-group

// Float64 partial q.k over dims 32p .. 32p+31 of one key: the four lanes of
// a quad (p = lane & 3) share a key, and quad_sum_f64 completes the sum.
// Every load of the lane is issued before its products.
template <bool KBF>
__device__ __forceinline__ double quad_dot_f64(const void* keys, size_t key_row,
                                               const float* __restrict__ qr, int p) {
  constexpr int D = saki::kHeadDim;
  float f[32], qv[32];
  if constexpr (KBF) {
    const uint4* kr = reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(keys) +
                                                     key_row * D + 32 * p);
#pragma unroll
    for (int u = 0; u < 4; ++u) unpack_piece<true>(kr[u], f + 8 * u);
  } else {
    const float4* kr = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(keys) +
                                                       key_row * D + 32 * p);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float4 v = kr[u];
      f[4 * u] = v.x; f[4 * u + 1] = v.y; f[4 * u + 2] = v.z; f[4 * u + 3] = v.w;
    }
  }
  const float4* q4 = reinterpret_cast<const float4*>(qr + 32 * p);
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const float4 v = q4[u];
    qv[4 * u] = v.x; qv[4 * u + 1] = v.y; qv[4 * u + 2] = v.z; qv[4 * u + 3] = v.w;
  }
  double a0 = 0.0, a1 = 0.0;
#pragma unroll
  for (int e = 0; e < 32; e += 2) {
    a0 = fma((double)qv[e], (double)f[e], a0);
    a1 = fma((double)qv[e + 1], (double)f[e + 1], a1);
  }
  return a0 + a1;
}
// The sum over the four lanes of a quad; every lane gets the same bits.
__device__ __forceinline__ double quad_sum_f64(double v) {
  v += __longlong_as_double((long long)xor_shfl_u64((uint64_t)__double_as_longlong(v), 1));
  return v + __longlong_as_double((long long)xor_shfl_u64((uint64_t)__double_as_longlong(v), 2));
}

// Exact top-k and recall hits in one scan.  A row's candidate list S (k
// distinct visible keys) gives the gate tau = min over S of a float32 lower
// bound of q.k; the scan collects C = {j : a3_j + E_j >= tau} with the bf16x3
// upper bound, so C contains the exact top-k T and, since every key of S
// passes, S as well.  Only the keys of C outside S (normally a handful) are
// rescored in float64.  Then, with |S| = k,
//   hits = |T intersect S| = k - |T intersect (C \ S)|,
// and a key o of C \ S is in T iff fewer than k keys of C beat it: the keys
// of S are compared through their float32 intervals (an undecided pair is
// settled in float64) and the others exactly.  With exact_idx or split keys
// the exact order is needed: S's keys in the chunk are rescored as well and
// merged with the others.  A row whose list is invalid (an entry outside
// [0, lim) or a duplicate) takes tau = -inf and treats all of C as others.
//
// A work-group of four waves owns 16 rows: the waves take four rows each for
// the gate and the final count, and every fourth key tile of the scan (all
// 16 rows, one collection list per wave and row, filled without atomics: the
// four lanes of a row append at offsets from a prefix of their counts), so
// that the latency of the per-row work is spread over four times as many
// waves.  A work-group in which one wave collects more than 64 keys for a
// row, or a row has more than 160 others, is flagged for exact_bf16_kernel.
// grid: 1-D xcd grid of ceil(Q / 16) * n_chunks * B * H_q work-groups; the
// flags use the numbering of the two-wave tiers.
template <bool KBF>
__global__ __launch_bounds__(kGateWaves * kWave) __attribute__((amdgpu_waves_per_eu(4))) void exact_gate_kernel(
    const void* __restrict__ keys, const uint8_t* __restrict__ khi,
    const uint8_t* __restrict__ klo, const float* __restrict__ knorm, const float* __restrict__ q,
    const int* __restrict__ q_pos, int H_q, int H_kv, int N_cap, int N_valid, int Q,
    int n_tiles_hi, int n_bh, int row_blocks2, int chunk, int n_chunks, int k,
    const int* __restrict__ approx, int* __restrict__ hits, int* __restrict__ exact_idx,
    KeyF64* __restrict__ part, int* __restrict__ redo) {
  constexpr int D = saki::kHeadDim;
  constexpr size_t TB = (size_t)kTile * D * 2;
  using KD = KeysF64;
  __shared__ int cj[kGateWaves][kMR * kGateRow];  // keys collected by each scanning wave
  __shared__ uint32_t sl[kMR * kWave];   // candidate lists, sorted descending
  __shared__ float ss[kMR * kWave];      // float32 score of sorted entry a
  __shared__ float se[kMR * kWave];      // and its error radius
  __shared__ float tau_s[kMR];           // gates
  __shared__ int bad_s[kMR];             // invalid lists
  __shared__ int ccount[kGateWaves][kMR];
  __shared__ int wg_fallback;
  __shared__ int bj_m[kGateWaves][kBatch];  // per wave: others' key, exact score, row
  __shared__ double bsc_m[kGateWaves][kBatch];
  __shared__ unsigned char brow_m[kGateWaves][kBatch];
  __shared__ int boff_m[kGateWaves][kMR / kGateWaves + 1];
  const int wave = threadIdx.x / kWave, lane = lane_id();
  const int row_blocks = (Q + kMR - 1) / kMR;
  const long long lb = xcd_logical_block((long long)row_blocks * n_chunks * n_bh);
  if (lb < 0) return;  // uniform over the work-group
  const int rb = (int)(lb % row_blocks), ch = (int)((lb / row_blocks) % n_chunks);
  const size_t bh = (size_t)(lb / ((long long)row_blocks * n_chunks));
  const int b = (int)(bh / H_q), h = (int)(bh % H_q);
  const int gkv = h / (H_q / H_kv);
  const size_t bg = (size_t)b * H_kv + gkv;
  const int row0 = rb * kMR;  // < Q
  const long long flag =
      (((long long)bh * n_chunks + ch) * row_blocks2 + rb / 2) * kMfmaWaves + (rb % 2);
  const int qi = lane % 16, g = lane / 16;
  const int my_row = row0 + qi;
  const bool row_ok = my_row < Q;
  const int my_lim = row_limit(my_row, Q, N_valid, q_pos);
  const int kmax = wave_max_i(my_lim);
  const int kbeg = ch * chunk;
  const int kend = min(kbeg + chunk, kmax);
  const int n_rows = min(kMR, Q - row0);
  const bool ordered = exact_idx != nullptr || n_chunks > 1;
  const size_t hoff = bg * n_tiles_hi * TB;
  const float* kn = knorm + bg * n_tiles_hi * kTile;
  const size_t kbase = bg * N_cap;
  int* bj = bj_m[wave];
  double* bsc = bsc_m[wave];
  unsigned char* brow = brow_m[wave];
  int* boff = boff_m[wave];

  // ---- gate, part 1: load, sort and check the candidate lists of rows wave,
  //      wave + 4, ... (the next row's list is loaded before this one is
  //      sorted); the owner wave also sets the row's gate to -inf and its
  //      validity flag (rows past Q count as invalid)
  {
    auto list_entry = [&](int r) -> int {
      return r < n_rows && lane < k ? approx[(bh * Q + row0 + r) * k + lane] : -1;
    };
    int aj_next = list_entry(wave);
#pragma unroll 1
    for (int r = wave; r < kMR; r += kGateWaves) {
      const int aj = aj_next;
      aj_next = list_entry(r + kGateWaves);
      if (lane == 0) tau_s[r] = -INFINITY;
      if (r >= n_rows) {
        if (lane == 0) bad_s[r] = 1;
        continue;
      }
      const int lim_r = __builtin_amdgcn_readlane(my_lim, r);
      bool bad = lane < k && (aj < 0 || aj >= lim_r);
      uint32_t key = lane < k ? (uint32_t)aj : (0x80000000u | (uint32_t)lane);
      wave_sort<KeysU32>(key);
      const uint32_t nxt = (uint32_t)__shfl_down((int)key, 1, kWave);
      bad |= lane < kWave - 1 && key == nxt;
      sl[r * kWave + lane] = key;
      if (lane == 0) bad_s[r] = __ballot(bad) != 0;  // an invalid list keeps tau = -inf
    }
  }
  if (threadIdx.x == 0) wg_fallback = 0;

  // query norm bound (lanes of row qi, dims 32kk + 8g .. +7); the MFMA
  // operands are formed after the gate
  const float* qrow = q + (bh * Q + (row_ok ? my_row : row0)) * D;  // a valid row
  float qn;
  {
    float sq = 0.f;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const float4 v0 = *reinterpret_cast<const float4*>(qrow + 32 * kk + 8 * g);
      const float4 v1 = *reinterpret_cast<const float4*>(qrow + 32 * kk + 8 * g + 4);
      sq = fmaf(v0.x, v0.x, sq); sq = fmaf(v0.y, v0.y, sq); sq = fmaf(v0.z, v0.z, sq); sq = fmaf(v0.w, v0.w, sq);
      sq = fmaf(v1.x, v1.x, sq); sq = fmaf(v1.y, v1.y, sq); sq = fmaf(v1.z, v1.z, sq); sq = fmaf(v1.w, v1.w, sq);
    }
    qn = row_ok ? sqrtf(sum_lane_groups(sq)) * (1.f + 1e-5f) : 0.f;
  }
  const float eq = kExactEps3 * qn;
  wave_lds_sync();

  // ---- gate, part 2: tau = min over the list of a float32 lower bound of q.k.
  //      Per row of the wave, eight steps of 8 sorted entries, 8 lanes per
  //      entry (dims 16p .. 16p+15), so each sum is at most 12 roundings deep
  //      (error <= gamma_12 ||q|| ||k||).  A row's entries and validity are
  //      read once; the steps take two key buffers in turn, each refilled
  //      right after use with the step two ahead (the next row's first two
  //      steps at the end of a row).  Pads (k < 64) and the entries of
  //      invalid lists read key 0 and are ignored.
  {
    const int p = lane & 7, slot = lane >> 3;
    const int my_rows_g = n_rows > wave ? (n_rows - wave + kGateWaves - 1) / kGateWaves : 0;
    // row rr of the wave: the key of entry 8u + slot in bit-free form (0 when
    // unused) and a bit mask of the used entries
    auto row_keys = [&](int rr, int (&jv)[8]) -> uint32_t {
      const int r = wave + kGateWaves * rr;
      const bool ok = bad_s[r] == 0;
      uint32_t used = 0;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint32_t kj = sl[r * kWave + 8 * u + slot];
        const bool use = ok && (kj >> 31) == 0;
        jv[u] = use ? (int)kj : 0;
        used |= use ? 1u << u : 0u;
      }
      return used;
    };
    // a key slice stays in its loaded form (four 16-byte words of float32,
    // or two of bf16) until it is used
    auto load_key = [&](uint4* w, float& knv, int j) {
      if constexpr (KBF) {
        const uint4* kr = reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(keys) +
                                                         (kbase + j) * D + 16 * p);
        w[0] = kr[0];
        w[1] = kr[1];
      } else {
        const uint4* kr = reinterpret_cast<const uint4*>(reinterpret_cast<const float*>(keys) +
                                                         (kbase + j) * D + 16 * p);
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) w[e4] = kr[e4];
      }
      knv = kn[j];
    };
    // the query slice of the wave's row rr (dims 16p .. 16p+15)
    auto load_q = [&](float* qv, int rr) {
      const float4* qr = reinterpret_cast<const float4*>(
          q + (bh * Q + row0 + wave + kGateWaves * rr) * D + 16 * p);
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const float4 v = qr[e4];
        qv[4 * e4] = v.x; qv[4 * e4 + 1] = v.y; qv[4 * e4 + 2] = v.z; qv[4 * e4 + 3] = v.w;
      }
    };
    // the key of entry 8u + slot of row rr if used, else -1
    auto entry_key = [&](int rr, int u) -> int {
      const int r = wave + kGateWaves * rr;
      const uint32_t kj = sl[r * kWave + 8 * u + slot];
      return bad_s[r] == 0 && (kj >> 31) == 0 ? (int)kj : -1;
    };
    if (my_rows_g > 0) {
      int jv[8];
      float qcur[16], qnext[16];
      uint4 ka[KBF ? 2 : 4], kb[KBF ? 2 : 4];
      float kna, knb;
      uint32_t used = row_keys(0, jv);
      load_q(qcur, 0);
      load_key(ka, kna, jv[0]);
      load_key(kb, knb, jv[1]);
      for (int rr = 0; rr < my_rows_g; ++rr) {
        const int r = wave + kGateWaves * rr;
        const bool more = rr + 1 < my_rows_g;
        // the next row's first two keys (pads and invalid lists read key 0)
        const int n0 = more ? max(entry_key(rr + 1, 0), 0) : 0;
        const int n1 = more ? max(entry_key(rr + 1, 1), 0) : 0;
        const float qr_n = readlane_s(qn, r);
        float lo = INFINITY;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (u == 4 && more) load_q(qnext, rr + 1);
          const uint4* w = (u & 1) ? kb : ka;
          const float knv = (u & 1) ? knb : kna;
          float f[16];
          if constexpr (KBF) {
            unpack_piece<true>(w[0], f);
            unpack_piece<true>(w[1], f + 8);
          } else {
#pragma unroll
            for (int e4 = 0; e4 < 4; ++e4) {
              f[4 * e4] = __uint_as_float(w[e4].x); f[4 * e4 + 1] = __uint_as_float(w[e4].y);
              f[4 * e4 + 2] = __uint_as_float(w[e4].z); f[4 * e4 + 3] = __uint_as_float(w[e4].w);
            }
          }
          float s0 = 0.f, s1 = 0.f;
#pragma unroll
          for (int e = 0; e < 16; e += 2) {
            s0 = fmaf(qcur[e], f[e], s0);
            s1 = fmaf(qcur[e + 1], f[e + 1], s1);
          }
          float sc = s0 + s1;
          sc += xor_shfl_f32(sc, 1);
          sc += xor_shfl_f32(sc, 2);
          sc += xor_shfl_f32(sc, 4);
          const float ea = kTauEps * qr_n * knv;
          const bool use = (used >> u) & 1u;
          if (use && p == 0) {
            ss[r * kWave + 8 * u + slot] = sc;
            se[r * kWave + 8 * u + slot] = ea;
          }
          lo = fminf(lo, use ? sc - ea : INFINITY);
          // refill this buffer with the step two ahead
          if (u + 2 < 8 || more) {
            const int j2 = u + 2 < 8 ? jv[u + 2] : (u == 6 ? n0 : n1);
            if (u & 1) load_key(kb, knb, j2);
            else load_key(ka, kna, j2);
          }
        }
        lo = wave_min_f32(lo);
        if (lane == 0 && bad_s[r] == 0) tau_s[r] = lo;
        if (more) {
          used = row_keys(rr + 1, jv);
#pragma unroll
          for (int e = 0; e < 16; ++e) qcur[e] = qnext[e];
        }
      }
    }
  }
  __syncthreads();

  // query MFMA operands: bf16 hi/lo split of dims 32kk + 8g .. +7
  bf16x8_t qh[4], ql[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    const float4 v0 = *reinterpret_cast<const float4*>(qrow + 32 * kk + 8 * g);
    const float4 v1 = *reinterpret_cast<const float4*>(qrow + 32 * kk + 8 * g + 4);
    const float fv[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
    float fh[8], fl[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float f = row_ok ? fv[e] : 0.f;
      fh[e] = bf16_round(f);
      fl[e] = bf16_round(f - fh[e]);
    }
    qh[kk] = as_bf16x8(pack_bf16x8(fh));
    ql[kk] = as_bf16x8(pack_bf16x8(fl));
  }

  // ---- scan (every fourth tile): collect the keys whose upper bound reaches
  //      the gate into this wave's lists; the four lanes of a row (lane
  //      groups g) append at offsets from a prefix of their counts
  int base = 0;  // this wave's entries for row qi so far (same in the row's four lanes)
  {
    const float my_tau = tau_s[qi];
    int* my_list = cj[wave] + qi * kGateRow;
    // a tile is 16 steps (sub-tile s, k-slice kk): each step's hi and lo
    // pieces come from a four-slot ring, refilled right after use with the
    // step four ahead (past the last tile: a repeat of a valid address)
    uint4 rh[4], rl[4];
    auto load_step = [&](int slot, int t0, int i) {
      const size_t o = hoff + (size_t)(t0 / kTile) * TB + (size_t)(4 * (i & 3) + g) * kTile * 16 +
                       (size_t)(16 * (i >> 2) + qi) * 16;
      rh[slot] = *reinterpret_cast<const uint4*>(khi + o);
      rl[slot] = *reinterpret_cast<const uint4*>(klo + o);
    };
    const int t_first = kbeg + wave * kTile;
    if (t_first < kend) {
#pragma unroll
      for (int i = 0; i < 4; ++i) load_step(i, t_first, i);
    }
    for (int t0 = t_first; t0 < kend; t0 += kGateWaves * kTile) {
      const int tn = t0 + kGateWaves * kTile < kend ? t0 + kGateWaves * kTile : t0;
      uint32_t take = 0;
#pragma unroll
      for (int sub = 0; sub < 4; ++sub) {
        const int kb = t0 + 16 * sub + 4 * g;
        const float4 nv = *reinterpret_cast<const float4*>(kn + kb);  // kb < n_tiles_hi * 64
        f32x4_t a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const int i = 4 * sub + kk;
          const bf16x8_t kh = as_bf16x8(rh[kk]), kl = as_bf16x8(rl[kk]);
          a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kh, qh[kk], a, 0, 0, 0);
          a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kl, qh[kk], a, 0, 0, 0);
          a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kh, ql[kk], a, 0, 0, 0);
          if (i + 4 < 16)
            load_step(kk, t0, i + 4);
          else
            load_step(kk, tn, i - 12);
        }
        const float nvs[4] = {nv.x, nv.y, nv.z, nv.w};
#pragma unroll
        for (int v = 0; v < 4; ++v)
          take |= (kb + v < my_lim && fmaf(eq, nvs[v], a[v]) >= my_tau) ? (1u << (4 * sub + v)) : 0u;
      }
      if (__ballot(take != 0) == 0) continue;
      const int c = __popc(take);
      const int c1 = (int)xor_shfl_u32((uint32_t)c, 16);   // count of lane group g ^ 1
      const int c2 = (int)xor_shfl_u32((uint32_t)c, 32);   // g ^ 2
      const int c3 = (int)xor_shfl_u32((uint32_t)c1, 32);  // g ^ 3
      // entries of the groups below g: g=1: g^1; g=2: g^2, g^3; g=3: g^3, g^2, g^1
      int pos = base + (g == 1 ? c1 : g == 2 ? c2 + c3 : g == 3 ? c1 + c2 + c3 : 0);
      base += c + c1 + c2 + c3;
#pragma unroll
      for (int sub = 0; sub < 4; ++sub)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (take & (1u << (4 * sub + v))) {
            my_list[min(pos, kGateCap)] = t0 + 16 * sub + 4 * g + v;
            ++pos;
          }
    }
  }
  if (lane < kMR) ccount[wave][lane] = base;  // lane r < 16 holds row r
  __syncthreads();
  bool fallback = __ballot(ccount[lane / kMR][lane % kMR] > kGateCap) != 0;

  // ---- rows wave, wave + 4, ...: the others C \ S, rescored in batches of whole rows
  int r_done = 0;  // of this wave's rows
  const int my_rows = n_rows > wave ? (n_rows - wave + kGateWaves - 1) / kGateWaves : 0;
  while (!fallback && r_done < my_rows) {
    int nb = 0, r_end = r_done;
    for (; r_end < my_rows; ++r_end) {
      const int r = wave + kGateWaves * r_end;
      const bool rbad = bad_s[r] != 0;
      // others of this row: all of C for an invalid list, else C minus S,
      // appended in one pass (entries past the batch are not written; a row
      // that does not fit is taken back and starts the next batch)
      const int nb0 = nb;
      int n_in_s = 0;
      for (int w = 0; w < kGateWaves; ++w) {
        const int c = ccount[w][r];
        for (int base = 0; base < c; base += kWave) {
          const int e = base + lane;
          const int j = e < c ? cj[w][r * kGateRow + e] : -1;
          const bool is_s = e < c && !rbad && in_sorted_desc(sl + r * kWave, j);
          const bool other = e < c && !is_s;
          const uint64_t m = __ballot(other);
          const int at = nb + prefix_count(m);
          if (other && at < kBatch) {
            bj[at] = j;
            brow[at] = (unsigned char)r;
          }
          nb += __popcll(m);
          n_in_s += __popcll(__ballot(is_s));
        }
      }
      // every key of a valid list passes the gate (a failed check means a bound
      // did not hold: hand the rows over rather than trust the result); a row
      // whose others do not fit one batch is handed over as well
      if ((!rbad && n_chunks == 1 && n_in_s != k) || nb - nb0 > kBatch) {
        fallback = true;
        break;
      }
      if (nb > kBatch) {  // this row starts the next batch
        nb = nb0;
        break;
      }
      if (lane == 0) {
        boff[r_end - r_done] = nb0;
        boff[r_end - r_done + 1] = nb;
      }
    }
    if (fallback) break;
    wave_lds_sync();

    // exact scores of the batch: four lanes per key, 16 keys per pass
    for (int base = 0; base < nb; base += kWave / 4) {
      const int e = base + lane / 4;
      const int ec = e < nb ? e : nb - 1;  // idle quads repeat the last key
      const size_t row = bh * Q + row0 + brow[ec];
      const double sx = quad_sum_f64(quad_dot_f64<KBF>(keys, kbase + bj[ec], q + row * D, lane & 3));
      if (e < nb && (lane & 3) == 0) bsc[e] = sx;
    }
    wave_lds_sync();

    // per row: the exact top-k decided by counting
    for (int rr = r_done; rr < r_end; ++rr) {
      const int r = wave + kGateWaves * rr;
      const size_t row = bh * Q + row0 + r;
      const float* qr = q + row * D;
      const bool rbad = bad_s[r] != 0;
      const int o0 = boff[rr - r_done], o1 = boff[rr - r_done + 1];
      // lane a: sorted list entry a (pads, k < 64, have the top bit set)
      const uint32_t kj = sl[r * kWave + lane];
      const bool real = (kj >> 31) == 0;
      const int aj = real ? (int)kj : -1;
      if (ordered) {
        KeyF64 xs = KD::pad();
        if (!rbad && real && aj >= kbeg && aj < kend)
          xs = KD::make(lane_dot_f64_g<KBF>(keys, kbase + aj, qr), aj);
        wave_sort<KD>(xs);
        for (int base = o0; base < o1; base += kWave) {
          KeyF64 xo = base + lane < o1 ? KD::make(bsc[base + lane], bj[base + lane]) : KD::pad();
          wave_sort<KD>(xo);
          wave_merge<KD>(xs, xo);
        }
        exact_row_out<KD>(xs, row, ch, n_chunks, k, approx, hits, exact_idx, part);
        continue;
      }
      // lane a: S's float32 interval of entry a
      const float sa = !rbad && real ? ss[r * kWave + lane] : 0.f;
      const float ea = !rbad && real ? se[r * kWave + lane] : 0.f;
      const double lo_a = (double)sa - (double)ea, hi_a = (double)sa + (double)ea;
      int in_t = 0, in_ts = 0;
      // others in blocks of 64, one per lane; the key compared with all of
      // them is read from its lane
      for (int base = o0; base < o1; base += kWave) {
        const int e = base + lane;
        const bool live = e < o1;
        const double so_l = live ? bsc[e] : 0.0;
        const int jo_l = live ? bj[e] : 0;
        int cnt = 0;  // keys of C that beat other e
        if (!rbad) {  // keys of S, through their intervals
          const int nbk = min(kWave, o1 - base);
          for (int t = 0; t < nbk; ++t) {
            const double so = readlane_s(so_l, t);
            const int jo = __builtin_amdgcn_readlane(jo_l, t);
            bool beat = real && lo_a > so;
            const bool amb = real && !beat && hi_a >= so;
            if (__ballot(amb) != 0 && amb) {
              const double sx = lane_dot_f64_g<KBF>(keys, kbase + aj, qr);
              beat = sx > so || (sx == so && aj < jo);
            }
            const int cs = __popcll(__ballot(beat));
            cnt += lane == t ? cs : 0;
          }
        }
        for (int base2 = o0; base2 < o1; base2 += kWave) {  // the other others, exactly
          const int e2 = base2 + lane;
          const double s2_l = base2 == base ? so_l : (e2 < o1 ? bsc[e2] : 0.0);
          const int j2_l = base2 == base ? jo_l : (e2 < o1 ? bj[e2] : 0);
          const int n2 = min(kWave, o1 - base2);
          for (int t = 0; t < n2; ++t) {
            const double s2 = readlane_s(s2_l, t);
            const int j2 = __builtin_amdgcn_readlane(j2_l, t);
            cnt += (s2 > so_l || (s2 == so_l && j2 < jo_l)) ? 1 : 0;
          }
        }
        const bool in = live && cnt < k;
        in_t += __popcll(__ballot(in));
        in_ts += __popcll(__ballot(in && rbad && in_sorted_desc(sl + r * kWave, jo_l)));
      }
      if (lane == 0) hits[row] = rbad ? in_ts : k - in_t;
    }
    wave_lds_sync();
    r_done = r_end;
  }
  if (fallback && lane == 0) atomicOr(&wg_fallback, 1);
  __syncthreads();
  if (threadIdx.x == 0) redo[flag] = wg_fallback;
}

// ---------------------------------------------------------------- merge of partials

// grid (rows), block 64 * waves (waves <= kMergeWaves): the waves of a row's
// work-group merge interleaved subsets of its sorted partial lists, then
// their lists are merged pairwise in a tree (wave w takes wave w + s's list at
// stride s = 1, 2, 4, ...).  RECALL: the row is an exact list -> exact_idx and
// hits.
// gates / redo: the gate check of score_scan_kernel's chunks (a row whose
// k-th score does not lie above every recorded gate gets redo = 1, else 0);
// only: merge just the rows flagged there.
constexpr int kMergeWaves = 16;

template <class KO, bool RECALL>
__global__ __launch_bounds__(kMergeWaves * kWave) void merge_kernel(
    const typename KO::K* __restrict__ part, size_t rows, int n_chunks, int k,
    int* __restrict__ out_idx, float* __restrict__ out_score,
    const int* __restrict__ approx, int* __restrict__ hits,
    const float* __restrict__ gates = nullptr, int* __restrict__ redo = nullptr,
    const int* __restrict__ only = nullptr) {
  using K = typename KO::K;
  __shared__ K lists[kMergeWaves][kWave];
  const int wave = threadIdx.x / kWave, lane = lane_id();
  const int waves = blockDim.x / kWave;
  const size_t row = blockIdx.x;
  if (row >= rows) return;
  if (only && only[row] == 0) return;  // the rows a rescan redid, nothing else
  // wave w merges partials w, w + waves, ..., eight at a time; the next
  // eight are loaded before the current ones are merged
  constexpr int kLoads = 8;
  K a = KO::pad();
  K nb[kLoads];
  auto load = [&](int c0) {
#pragma unroll
    for (int u = 0; u < kLoads; ++u) {
      const int c = c0 + u * waves;
      nb[u] = c < n_chunks ? part[(row * n_chunks + c) * kMaxK + lane] : KO::pad();
    }
  };
  if (wave < n_chunks) load(wave);
  for (int c0 = wave; c0 < n_chunks; c0 += kLoads * waves) {
    K b[kLoads];
#pragma unroll
    for (int u = 0; u < kLoads; ++u) b[u] = nb[u];
    if (c0 + kLoads * waves < n_chunks) load(c0 + kLoads * waves);
#pragma unroll
    for (int u = 0; u < kLoads; ++u)
      // a partial is sorted: skip it when its best cannot enter the list
      if (KO::gt(KO::readlane(b[u], 0), KO::readlane(a, kWave - 1))) wave_merge<KO>(a, b[u]);
  }
  lists[wave][lane] = a;
  __syncthreads();
  for (int st = 1; st < waves; st *= 2) {  // uniform trip count: every wave reaches each barrier
    const bool active = wave % (2 * st) == 0 && wave + st < waves;
    if (active) {
      const K b = lists[wave + st][lane];
      if (KO::gt(KO::readlane(b, 0), KO::readlane(a, kWave - 1))) wave_merge<KO>(a, b);
    }
    __syncthreads();
    if (active) lists[wave][lane] = a;
    __syncthreads();
  }
  if (wave != 0) return;
  const int j = out_index<KO>(a);
  if constexpr (RECALL) {
    if (out_idx && lane < k) out_idx[row * k + lane] = j;
    const int hsum = row_hits(j, approx, row, k);
    if (lane == 0) hits[row] = hsum;
  } else {
    if (lane < k) {
      out_idx[row * k + lane] = j;
      if (out_score) out_score[row * k + lane] = (float)KO::score(a);
    }
    if (gates) {  // score_scan_kernel's chunks that kept only the keys above a gate
      float gmax = -INFINITY;
      for (int c = lane; c < n_chunks; c += kWave) gmax = fmaxf(gmax, gates[row * n_chunks + c]);
      gmax = wave_max_f32(gmax);
      // exact when every recorded gate lies below the k-th score: keys a gate
      // left out score at most the gate
      const float sk = (float)KO::score(KO::readlane(a, k - 1));
      if (lane == 0) redo[row] = (gmax == -INFINITY || sk > gmax) ? 0 : 1;
    }
  }
}

// ---------------------------------------------------------------- calibration moments

// grid: (H_q + H_kv) * nb * (nb + 1) / 2 work-groups, nb = ceil(d / 64), block
// 256.  Work-group (head, block pair bi <= bj) forms the 64 x 64 block (rows
// 64 bi.., columns 64 bj..) of that head's moment and writes it and its
// mirror: thread (ty, tx) holds the 4 x 4 outputs of rows 64 bi + 4 ty ..,
// columns 64 bj + 4 tx .., each a float64 sum over the tokens in order.
// Heads below H_q are query heads (uncentred); the rest are KV heads, centred
// by their column means, which every work-group computes for its own 128
// columns.  Tokens are staged in LDS 32 at a time.
constexpr int kMomBlk = 64;
constexpr int kMomChunk = 32;  // tokens staged per step

__global__ __launch_bounds__(256) void moments_kernel(const float* __restrict__ q_cal,
                                                      const float* __restrict__ k_cal, int H_q,
                                                      int T, int d, double* __restrict__ Sq,
                                                      double* __restrict__ Sk,
                                                      double* __restrict__ mu_out) {
  const int nb = (d + kMomBlk - 1) / kMomBlk;
  const int npairs = nb * (nb + 1) / 2;
  const int head = blockIdx.x / npairs;
  int bi = 0, rem = blockIdx.x % npairs;  // the pair's rank in row-major order of bi <= bj
  while (rem >= nb - bi) {
    rem -= nb - bi;
    ++bi;
  }
  const int bj = bi + rem;
  const bool key = head >= H_q;
  const int hh = key ? head - H_q : head;
  const float* X = (key ? k_cal : q_cal) + (size_t)hh * T * d;
  const int tid = threadIdx.x;
  const int tx = tid % 16, ty = tid / 16;
  const int i0 = bi * kMomBlk, j0 = bj * kMomBlk;
  __shared__ double xi[kMomChunk][kMomBlk], xj[kMomChunk][kMomBlk];
  __shared__ double mean[2 * kMomBlk];
  __shared__ double part[2][2 * kMomBlk];
  // column means (KV heads): two threads per column, even and odd tokens
  {
    const int c = tid % (2 * kMomBlk), h = tid / (2 * kMomBlk);
    const int col = c < kMomBlk ? i0 + c : j0 + c - kMomBlk;
    double m = 0.0;
    if (key && col < d) {
#pragma unroll 16
      for (int t = h; t < T; t += 2) m += (double)X[(size_t)t * d + col];
    }
    part[h][c] = m;
  }
  __syncthreads();
  if (tid < 2 * kMomBlk) mean[tid] = key ? (part[0][tid] + part[1][tid]) / (double)T : 0.0;
  __syncthreads();
  double acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[a][e] = 0.0;
  // tokens t0 .. t0 + 31 of both column blocks: element u of this thread is
  // token t0 + (tid + 256 u) / 64, column (tid + 256 u) % 64; the next chunk's
  // values are loaded while this one is summed
  constexpr int kPer = kMomChunk * kMomBlk / 256;
  float ni[kPer], nj[kPer];
  auto load_chunk = [&](int t0) {
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int e = tid + 256 * u, t = t0 + e / kMomBlk, c = e % kMomBlk;
      ni[u] = (t < T && i0 + c < d) ? X[(size_t)t * d + i0 + c] : 0.f;
      nj[u] = (t < T && j0 + c < d) ? X[(size_t)t * d + j0 + c] : 0.f;
    }
  };
  load_chunk(0);
  for (int t0 = 0; t0 < T; t0 += kMomChunk) {
    // stage the chunk (centred; 0 past T or d), then request the next one
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int e = tid + 256 * u, tt = e / kMomBlk, c = e % kMomBlk, t = t0 + tt;
      xi[tt][c] = (t < T && i0 + c < d) ? (double)ni[u] - mean[c] : 0.0;
      xj[tt][c] = (t < T && j0 + c < d) ? (double)nj[u] - mean[kMomBlk + c] : 0.0;
    }
    if (t0 + kMomChunk < T) load_chunk(t0 + kMomChunk);
    __syncthreads();
#pragma unroll 4
    for (int tt = 0; tt < kMomChunk; ++tt) {
      double va[4], vb[4];
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        va[a] = xi[tt][4 * ty + a];
        vb[a] = xj[tt][4 * tx + a];
      }
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[a][e] = fma(va[a], vb[e], acc[a][e]);
    }
    __syncthreads();
  }
  double* S = key ? Sk + (size_t)hh * d * d : Sq + (size_t)hh * d * d;
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int i = i0 + 4 * ty + a, j = j0 + 4 * tx + e;
      if (i < d && j < d) {
        const double v = acc[a][e] / (double)T;
        S[(size_t)i * d + j] = v;
        S[(size_t)j * d + i] = v;
      }
    }
  if (key && bi == 0 && tid < kMomBlk && j0 + tid < d) mu_out[(size_t)hh * d + j0 + tid] = mean[kMomBlk + tid];
}

// ---------------------------------------------------------------- reading the winners

__device__ __forceinline__ float wave_sum_f32(float v) {
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) v += xor_shfl_f32(v, m);
  return v;
}

// sin and cos of pos * inv (radians): the product and its reduction to
// [-pi, pi] in float64, the functions in float32.
__device__ __forceinline__ void rope_sincos(int pos, double inv, float* s, float* c) {
  constexpr double kTwoPi = 6.283185307179586476925286766559;
  const double a = (double)pos * inv;
  const float red = (float)(a - kTwoPi * rint(a / kTwoPi));
  sincosf(red, s, c);
}

constexpr int kAttendWaves = 4;   // waves per row
constexpr int kAttendBatch = 16;  // list entries per wave: wave w takes 16w .. 16w + 15

// grid (Q, B * H_q), block 256: one work-group per (sequence, head, query)
// row, k <= 64.  Lane l holds dims l and l + 64 of the rotated query and of
// each key, so that the RoPE pairs (m, m + d/2) stay inside a lane, and a
// key's score is a wave sum.  Each wave gathers its 16 entries' keys (or, for
// reconstruction, unpacks their codes into LDS and forms mu + B_q c) and
// values in one round of loads, and keeps the softmax of its entries relative
// to its own maximum; the four partial results are then rescaled to the
// row's maximum and added.
template <int RK, bool KBF, int ST, bool RECON>
__global__ __launch_bounds__(kAttendWaves * kWave) void attend_kernel(
    const void* __restrict__ keys, const float* __restrict__ values,
    const uint8_t* __restrict__ index, int n_tiles, int H_q, int H_kv, int index_heads,
    int N_cap, int N_valid, const float* __restrict__ q, const int* __restrict__ q_pos, int Q,
    const float* __restrict__ Bq, const float* __restrict__ mu,
    const int* __restrict__ top_idx, int k, float log_theta, float* __restrict__ out) {
  constexpr int D = saki::kHeadDim;
  constexpr int HALF = D / 2;
  static_assert(HALF == kWave, "one RoPE pair per lane");
  static_assert(kAttendWaves * kAttendBatch == kWave, "the waves cover a 64-entry list");
  constexpr int ES = code_bytes<ST>();
  constexpr int CPP = saki::kChunkBytes / ES;
  constexpr int NP = RK / CPP;
  constexpr size_t TB = (size_t)kTile * RK * ES;
  __shared__ float bq_s[RECON ? D : 1][RECON ? RK + 1 : 1];
  __shared__ float code_s[kAttendWaves][RECON ? kAttendBatch : 1][RECON ? RK : 1];
  __shared__ float part_m[kAttendWaves], part_l[kAttendWaves];
  __shared__ float part_o[kAttendWaves][D];
  const int wave = threadIdx.x / kWave, lane = lane_id();
  const int i = blockIdx.x;
  const size_t bh = blockIdx.y;
  const int h = (int)(bh % H_q);
  const size_t b = bh / H_q;
  const int g = h / (H_q / H_kv);
  const size_t row = bh * Q + i;
  const size_t kbase = ((size_t)b * H_kv + g) * N_cap;
  const size_t cset = b * index_heads + h / (H_q / index_heads);
  const int e0 = wave * kAttendBatch;
  // lane u < 16: list entry e0 + u (-1 past k)
  const int my_j = lane < kAttendBatch && e0 + lane < k ? top_idx[row * k + e0 + lane] : -1;
  if constexpr (RECON) {
    for (int e = threadIdx.x; e < D * RK; e += blockDim.x)
      bq_s[e / RK][e % RK] = Bq[(size_t)h * D * RK + e];
  }
  const double inv = exp(-(2.0 * lane / D) * (double)log_theta);  // theta^(-2l/d)
  float qa, qb;
  {
    float sn, cs;
    rope_sincos(q_pos ? q_pos[i] : N_valid - 1, inv, &sn, &cs);
    const float a0 = q[row * D + lane], a1 = q[row * D + lane + HALF];
    qa = a0 * cs - a1 * sn;
    qb = a1 * cs + a0 * sn;
  }
  int jj[kAttendBatch];
#pragma unroll
  for (int u = 0; u < kAttendBatch; ++u) {
    const int j = __builtin_amdgcn_readlane(my_j, u);
    jj[u] = j < N_valid ? j : -1;  // entries outside [0, N_valid) are skipped
  }
  // keys (or codes) and values of the wave's entries; a skipped entry reads
  // row 0 and gets weight 0
  float k0[kAttendBatch], k1[kAttendBatch], v0[kAttendBatch], v1[kAttendBatch];
#pragma unroll
  for (int u = 0; u < kAttendBatch; ++u) {
    const size_t kr = (kbase + (size_t)max(jj[u], 0)) * D;
    v0[u] = values[kr + lane];
    v1[u] = values[kr + lane + HALF];
    if constexpr (!RECON) {
      k0[u] = load_key_elem<KBF>(keys, kr + lane);
      k1[u] = load_key_elem<KBF>(keys, kr + lane + HALF);
    }
  }
  if constexpr (RECON) {
    for (int t0 = 0; t0 < kAttendBatch * NP; t0 += kWave) {
      // lane t0 + lane unpacks piece p of entry u; the entry is read from
      // its lane by every lane of the wave (all lanes active)
      const int t = t0 + lane;
      const int u = min(t / NP, kAttendBatch - 1), p = t % NP;
      int j = __shfl(my_j, u, kWave);
      j = j >= 0 && j < N_valid ? j : 0;
      if (t < kAttendBatch * NP) {
        const uint4 v = *reinterpret_cast<const uint4*>(
            index + (cset * n_tiles + j / kTile) * TB + (size_t)p * kTile * 16 + (size_t)(j % kTile) * 16);
        float f[CPP];
        unpack_codes<ST>(v, f);
#pragma unroll
        for (int c = 0; c < CPP; ++c) code_s[wave][u][p * CPP + c] = f[c];
      }
    }
    __syncthreads();  // B_q staged by the work-group, codes by the wave
    const float mu0 = mu[(size_t)g * D + lane], mu1 = mu[(size_t)g * D + lane + HALF];
#pragma unroll
    for (int u = 0; u < kAttendBatch; ++u) {
      k0[u] = mu0;
      k1[u] = mu1;
    }
#pragma unroll 2
    for (int m = 0; m < RK; ++m) {  // k_hat = mu + B_q c, one code element of all 16 keys at a time
      const float b0 = bq_s[lane][m], b1 = bq_s[lane + HALF][m];
#pragma unroll
      for (int u = 0; u < kAttendBatch; ++u) {
        const float cv = code_s[wave][u][m];
        k0[u] = fmaf(b0, cv, k0[u]);
        k1[u] = fmaf(b1, cv, k1[u]);
      }
    }
  }
  float my_s = -INFINITY;  // lane u: score of entry e0 + u
#pragma unroll
  for (int u = 0; u < kAttendBatch; ++u) {
    float sn, cs;
    rope_sincos(max(jj[u], 0), inv, &sn, &cs);
    const float kb0 = k0[u] * cs - k1[u] * sn, kb1 = k1[u] * cs + k0[u] * sn;
    const float sc = wave_sum_f32(fmaf(qa, kb0, qb * kb1)) * (1.f / 11.313708498984761f);
    if (lane == u && jj[u] >= 0) my_s = sc;
  }
  // this wave's softmax terms relative to its own maximum
  const float mx = wave_max_f32(my_s);
  const float pw = my_s == -INFINITY ? 0.f : expf(my_s - mx);
  const float l = wave_sum_f32(pw);
  float o0 = 0.f, o1 = 0.f;
#pragma unroll
  for (int u = 0; u < kAttendBatch; ++u) {
    const float pe = readlane_s(pw, u);
    o0 = fmaf(pe, v0[u], o0);
    o1 = fmaf(pe, v1[u], o1);
  }
  if (lane == 0) {
    part_m[wave] = mx;
    part_l[wave] = l;
  }
  part_o[wave][lane] = o0;
  part_o[wave][lane + HALF] = o1;
  __syncthreads();
  if (wave != 0) return;
  // rescale to the row's maximum and add (an empty row writes zeros)
  float M = -INFINITY;
#pragma unroll
  for (int w = 0; w < kAttendWaves; ++w) M = fmaxf(M, part_m[w]);
  float L = 0.f, a0 = 0.f, a1 = 0.f;
#pragma unroll
  for (int w = 0; w < kAttendWaves; ++w) {
    const float f = part_m[w] == -INFINITY ? 0.f : expf(part_m[w] - M);
    L = fmaf(f, part_l[w], L);
    a0 = fmaf(f, part_o[w][lane], a0);
    a1 = fmaf(f, part_o[w][lane + HALF], a1);
  }
  const float il = L > 0.f ? 1.f / L : 0.f;
  out[row * D + lane] = a0 * il;
  out[row * D + lane + HALF] = a1 * il;
}

template <int RK, bool KBF, int ST, bool RECON>
void launch_attend(const void* keys, const float* values, const uint8_t* index, int B, int H_q,
                   int H_kv, int index_heads, int N_cap, int N_valid, const float* q,
                   const int* q_pos, int Q, const float* Bq, const float* mu, const int* top_idx,
                   int k, float rope_theta, float* out, hipStream_t s) {
  dim3 grid((unsigned)Q, (unsigned)(B * H_q));
  hipLaunchKernelGGL((attend_kernel<RK, KBF, ST, RECON>), grid, dim3(kAttendWaves * kWave), 0, s,
                     keys, values, index, (int)saki::n_tiles(N_cap), H_q, H_kv, index_heads, N_cap,
                     N_valid, q, q_pos, Q, Bq, mu, top_idx, k, logf(rope_theta), out);
}

// ---------------------------------------------------------------- dispatch helpers

bool launch_ok() { return hipGetLastError() == hipSuccess; }

// 1-D grid for xcd_logical_block: 8 * ceil(total / 8) work-groups.
dim3 xcd_grid(const saki::Plan& p, int n_bh) {
  const long long total = (long long)p.row_blocks * p.n_chunks * n_bh;
  return dim3((unsigned)(((total + kXcds - 1) / kXcds) * kXcds));
}

// Work-groups of `kernel` (block `threads`) resident on the whole current
// device at once, or 0 if the runtime cannot tell.  Cached per (kernel,
// block size, device).
template <class K>
int resident_groups(K kernel, int threads) {
  static std::mutex mu;
  static std::map<std::tuple<const void*, int, int>, int> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  const auto key = std::make_tuple(reinterpret_cast<const void*>(kernel), threads, dev);
  {
    std::lock_guard<std::mutex> lock(mu);
    const auto it = cache.find(key);
    if (it != cache.end()) return it->second;
  }
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  std::lock_guard<std::mutex> lock(mu);
  cache[key] = cus * per_cu;
  return cus * per_cu;
}

template <int RK, bool KBF, int ST>
void launch_build(const void* keys, const float* Bk, const float* mu, int B, int H_q,
                  int H_kv, int N_cap, uint8_t* index, int n_begin, int n_end,
                  hipStream_t s) {
  const int k0 = (n_begin / 16) * 16;
  const int per_head = n_end - n_begin <= kBuildSplitKeys ? 1 : 0;
  const long long units = (long long)(per_head ? H_q : H_kv) * B;
  // slices of at least kBuildKeys keys, about as many work-groups as the
  // device holds at once
  int slices = (n_end - k0 + kBuildKeys - 1) / kBuildKeys;
  if (!per_head) {
    const int slots = resident_groups(build_index_kernel<RK, KBF, ST>, kBuildWaves * kWave);
    if (slots > 0) slices = (int)std::max(1LL, std::min((long long)slices, kBuildRounds * slots / units));
  }
  dim3 grid(slices, per_head ? H_q : H_kv, B);
  hipLaunchKernelGGL((build_index_kernel<RK, KBF, ST>), grid, dim3(kBuildWaves * kWave), 0, s, keys, Bk, mu, H_q,
                     H_kv, N_cap, (int)saki::n_tiles(N_cap), index, n_begin, n_end, per_head);
}

// A split-N streaming launch that fills the GPU exactly once: the plan's
// chunking (which sized the workspace) is coarsened so that the work-groups
// number at most what the device holds at one time (or, given
// max_waves_per_simd, at most that many waves per SIMD), the chunk count
// staying within the plan's.  A work-group takes `chunks_per_group` chunks.
template <class K>
saki::Plan one_round(saki::Plan p, K kernel, int groups_per_chunk, int chunks_per_group,
                     int N_valid, int max_waves_per_simd = 0) {
  if (p.n_chunks <= 1) return p;
  int slots = resident_groups(kernel, kWave * p.waves);
  if (max_waves_per_simd > 0 && slots > 0) {  // at most this many waves on each of a CU's 4 SIMDs
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess)
      slots = min(slots, cus * 4 * max_waves_per_simd / p.waves);
  }
  if (slots <= 0) return p;
  const int want = max(1, slots / max(1, groups_per_chunk)) * chunks_per_group;
  const size_t n = N_valid > 0 ? (size_t)N_valid : 1;
  size_t chunk = saki::round_up((n + want - 1) / want, kTile);
  const int n_chunks = (int)((n + chunk - 1) / chunk);
  if (n_chunks >= p.n_chunks) return p;
  p.chunk = (int)chunk;
  p.n_chunks = n_chunks;
  return p;
}

template <int RK, int ST>
void launch_score(const uint8_t* index, int B, int H_q, int H_kv, int index_heads, int N_cap,
                  int N_valid, const float* q, const int* q_pos, int Q, const float* Bq,
                  const float* mu, int k, int* top_idx, float* top_score, uint8_t* ws,
                  const saki::Plan& p0, hipStream_t s) {
  const int gq = H_q / index_heads;
  saki::Plan p = p0;
  if (p.scan) {
    const long long wr = p0.row_blocks, per_chunk = wr * B * H_q;
    // two waves per SIMD: VALU-heavy waves of equal work, none waiting on a third
    p = one_round(p0, score_scan_kernel<RK, ST>, (int)((per_chunk + kScanWaves - 1) / kScanWaves), 1,
                  N_valid, 2);
    const int nt = (int)saki::n_tiles(N_cap);
    auto launch = [&](int chunk, int n_chunks, uint64_t* part, float* gates, const int* only) {
      const long long groups = (per_chunk * n_chunks + kScanWaves - 1) / kScanWaves;
      hipLaunchKernelGGL((score_scan_kernel<RK, ST>), dim3((unsigned)(((groups + kXcds - 1) / kXcds) * kXcds)),
                         dim3(kScanWaves * kWave), 0, s, index, nt, N_valid, Q, q_pos, q, Bq, mu, H_q,
                         H_kv, gq, B * H_q, (int)wr, chunk, n_chunks, k, top_idx, top_score, part,
                         gates, only);
    };
    if (p.n_chunks == 1) {
      launch(p.chunk, 1, nullptr, nullptr, nullptr);
      return;
    }
    // chunks, their merge with the gate check, then the flagged rows over all keys
    uint64_t* part = reinterpret_cast<uint64_t*>(ws + p.part_off);
    float* gates = reinterpret_cast<float*>(ws + p.z_off);
    int* redo = reinterpret_cast<int*>(ws + p.flag_off);
    launch(p.chunk, p.n_chunks, part, gates, nullptr);
    const size_t rows = (size_t)B * H_q * Q;
    // one wave per row: its loads of eight partial lists at a time are in
    // flight together, and few chunks leave little to split further
    hipLaunchKernelGGL((merge_kernel<KeysF32, false>), dim3((unsigned)rows), dim3(kWave), 0, s, part,
                       rows, p.n_chunks, k, top_idx, top_score, nullptr, nullptr, gates, redo);
    // the flagged rows' chunks again without a gate, and their merge
    launch(p.chunk, p.n_chunks, part, gates, redo);
    hipLaunchKernelGGL((merge_kernel<KeysF32, false>), dim3((unsigned)rows), dim3(kWave), 0, s, part,
                       rows, p.n_chunks, k, top_idx, top_score, nullptr, nullptr, nullptr, nullptr,
                       redo);
    return;
  }
  const int cpg = p0.split ? p0.waves : 1;  // chunks per work-group
  if (!p.mfma)
    p = p.rows == 4 ? one_round(p0, score_stream_kernel<RK, ST, 4>, p0.row_blocks * B * index_heads, cpg, N_valid)
                    : one_round(p0, score_stream_kernel<RK, ST, 1>, p0.row_blocks * B * index_heads, cpg, N_valid);
  const size_t rows = (size_t)B * H_q * Q;
  uint64_t* part = p.n_chunks > 1 ? reinterpret_cast<uint64_t*>(ws + p.part_off) : nullptr;
  dim3 grid((unsigned)(p.row_blocks * ((p.n_chunks + cpg - 1) / cpg)), B * index_heads);
  dim3 block(kWave * p.waves);
  const int nt = (int)saki::n_tiles(N_cap);
  if (p.mfma) {
    uint8_t* zq = ws + p.z_off;
    float* zb = reinterpret_cast<float*>(ws + p.b_off);
    const int parts = (Q + kQsRows - 1) / kQsRows;
    const long long qs_groups = (long long)parts * B * H_q;
    hipLaunchKernelGGL((query_sketch_kernel<RK, ST>), dim3((unsigned)(((qs_groups + kXcds - 1) / kXcds) * kXcds)),
                       dim3(kQsWaves * kWave), 0, s, q, Bq, mu, Q, H_q, H_kv, B * H_q, parts, zq, zb);
    hipLaunchKernelGGL((score_batch_kernel<RK, ST>), xcd_grid(p, B * H_q), dim3(kBWaves * kWave), 0,
                       s, index, nt, N_valid, Q, q_pos, zq, zb, H_q, gq, B * H_q,
                       p.row_blocks, p.chunk, p.n_chunks, k, top_idx, top_score, part);
  }
  else if (p.rows == 4)
    hipLaunchKernelGGL((score_stream_kernel<RK, ST, 4>), grid, block, 0, s, index, nt, N_valid,
                       Q, q_pos, q, Bq, mu, H_q, H_kv, gq, p.row_blocks, p.chunk, p.n_chunks,
                       (int)p.split, k, top_idx, top_score, part);
  else
    hipLaunchKernelGGL((score_stream_kernel<RK, ST, 1>), grid, block, 0, s, index, nt, N_valid,
                       Q, q_pos, q, Bq, mu, H_q, H_kv, gq, p.row_blocks, p.chunk, p.n_chunks,
                       (int)p.split, k, top_idx, top_score, part);
  if (p.n_chunks > 1)
    hipLaunchKernelGGL((merge_kernel<KeysF32, false>), dim3((unsigned)rows),
                       dim3(kWave * min(kMergeWaves, p.n_chunks)), 0, s, part, rows, p.n_chunks,
                       k, top_idx, top_score, nullptr, nullptr);
}

template <bool KBF>
void launch_recall(const void* keys, const float* q, const int* q_pos, int B, int H_q,
                   int H_kv, int N_cap, int N_valid, int Q, int k, const int* approx,
                   int* hits, int* exact_idx, uint8_t* ws, const saki::Plan& p,
                   hipStream_t s) {
  const size_t rows = (size_t)B * H_q * Q;
  KeyF64* part = p.n_chunks > 1 ? reinterpret_cast<KeyF64*>(ws + p.part_off) : nullptr;
  dim3 grid((unsigned)(p.row_blocks * p.n_chunks), B * H_q);
  dim3 block(kWave * p.waves);
  if (p.mfma) {
    const int nt_hi = (int)saki::n_tiles(N_valid);
    uint8_t* khi = ws + p.z_off;
    uint8_t* klo = khi + (size_t)B * H_kv * nt_hi * kTile * saki::kHeadDim * 2;
    float* knorm = reinterpret_cast<float*>(ws + p.b_off);
    // three tiers, each running only the waves the previous one flagged
    int* flag1 = reinterpret_cast<int*>(ws + p.flag_off);
    int* flag2 = flag1 + p.flag_count;
    if (nt_hi > 0)
      hipLaunchKernelGGL((keys_hi_kernel<KBF>), dim3(nt_hi, B * H_kv), dim3(256), 0, s, keys, N_cap,
                         N_valid, nt_hi, khi, klo, knorm);
    {
      const long long total = (long long)((Q + kMR - 1) / kMR) * p.n_chunks * B * H_q;
      hipLaunchKernelGGL((exact_gate_kernel<KBF>), dim3((unsigned)(((total + kXcds - 1) / kXcds) * kXcds)),
                         dim3(kGateWaves * kWave), 0, s, keys, khi, klo, knorm, q, q_pos, H_q, H_kv, N_cap,
                         N_valid, Q, nt_hi, B * H_q, p.row_blocks, p.chunk, p.n_chunks, k, approx,
                         hits, exact_idx, part, flag1);
    }
    hipLaunchKernelGGL((exact_bf16_kernel<KBF>), xcd_grid(p, B * H_q), block, 0, s, keys, khi,
                       klo, knorm, q, q_pos, H_q, H_kv, N_cap, N_valid, Q, nt_hi, B * H_q,
                       p.row_blocks, p.chunk, p.n_chunks, k, approx, hits, exact_idx, part,
                       (const int*)flag1, flag2);
    hipLaunchKernelGGL((exact_mfma_kernel<KBF>), xcd_grid(p, B * H_q), block, 0, s, keys, q,
                       q_pos, H_q, H_kv, N_cap, N_valid, Q, p.row_blocks, p.chunk, p.n_chunks, k,
                       approx, hits, exact_idx, part, B * H_q, (const int*)flag2);
  } else if (p.rows == 4) {
    hipLaunchKernelGGL((exact_stream_kernel<KBF, 4>), grid, block, 0, s, keys, q, q_pos, H_q,
                       H_kv, N_cap, N_valid, Q, p.row_blocks, p.chunk, p.n_chunks, k, approx,
                       hits, exact_idx, part);
  } else {
    hipLaunchKernelGGL((exact_stream_kernel<KBF, 1>), grid, block, 0, s, keys, q, q_pos, H_q,
                       H_kv, N_cap, N_valid, Q, p.row_blocks, p.chunk, p.n_chunks, k, approx,
                       hits, exact_idx, part);
  }
  if (p.n_chunks > 1)
    hipLaunchKernelGGL((merge_kernel<KeysF64, true>), dim3((unsigned)rows),
                       dim3(kWave * min(kMergeWaves, p.n_chunks)), 0, s, part, rows, p.n_chunks,
                       k, exact_idx, nullptr, approx, hits);
}

bool dtype_ok(int t) { return t == SAKI_F32 || t == SAKI_BF16; }  // keys
bool sketch_ok(int t) { return t == SAKI_F32 || t == SAKI_BF16 || t == SAKI_FP8; }

// Common size validation of the GPU entry points.
int check_common(int B, int H_q, int H_kv, int N_cap, int N_valid, int d) {
  if (B <= 0 || H_q <= 0 || H_kv <= 0 || H_q % H_kv != 0 || N_cap < 0 || N_valid < 0 ||
      N_valid > N_cap || d <= 0)
    return SAKI_ERR_ARG;
  if (B > 65535 || (long long)B * H_q > 65535) return SAKI_ERR_UNSUPPORTED;
  if (d != saki::kHeadDim) return SAKI_ERR_UNSUPPORTED;
  return SAKI_OK;
}

// Scratch memory of the allocation-free score entry point: a static device
// array, one copy per GPU the library runs on (held until the process
// ends).  In host code `scratch` names a host-side stand-in, never the
// device memory: the device address comes from hipGetSymbolAddress, taken
// once per device with that device current, and only that address is
// passed to kernels.
constexpr size_t kScratchBytes = (size_t)32 << 20;

}  // namespace

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void* scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array (*out), or an error.
int scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return SAKI_ERR_HIP;
  }
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
      (void)hipGetLastError();
      return SAKI_ERR_HIP;
    }
    scratch_ptr[dev] = ptr;
  }
  *out = scratch_ptr[dev];
  return SAKI_OK;
}

// saki_score_topk with ws == NULL meaning the static scratch array (whose
// size the caller passes as ws_bytes).
int score_topk_impl(const void* index, int sketch_dtype, int B, int H_q, int H_kv,
                    int index_heads, int N_cap, int N_valid, int d, int r, const float* q,
                    const int* q_pos, int Q, const float* B_q, const float* mu, int k,
                    int* top_idx, float* top_score, void* ws, size_t ws_bytes, void* stream) {
  int st = check_common(B, H_q, H_kv, N_cap, N_valid, d);
  if (st != SAKI_OK) return st;
  if (Q < 0) return SAKI_ERR_ARG;
  // a code set serves whole query heads and lies within one KV group
  if (index_heads <= 0 || H_q % index_heads != 0 || index_heads % H_kv != 0) return SAKI_ERR_ARG;
  if (!sketch_ok(sketch_dtype) || !saki::rank_supported(r) || k < 1 || k > kMaxK)
    return SAKI_ERR_UNSUPPORTED;
  if (Q == 0) return SAKI_OK;
  if (!index || !q || !B_q || !mu || !top_idx) return SAKI_ERR_ARG;
  const saki::Plan p = saki::score_plan(B, H_q, index_heads, Q, N_valid, r, sketch_dtype);
  if (ws_bytes < p.ws_bytes) return SAKI_ERR_WORKSPACE;
  if (!ws) {  // the static scratch array, resolved only once the sizes fit it
    const int sst = scratch_address(&ws);
    if (sst != SAKI_OK) return sst;
  }
  if ((size_t)p.row_blocks * p.n_chunks > 0x7fffffffu) return SAKI_ERR_UNSUPPORTED;
  // the one-pass kernel's 1-D grid: one wave per (head, row block, chunk)
  if (p.scan && (size_t)B * H_q * p.row_blocks * p.n_chunks * kWave >= 0xffffffffu)
    return SAKI_ERR_UNSUPPORTED;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const uint8_t* ix = reinterpret_cast<const uint8_t*>(index);
  uint8_t* w = reinterpret_cast<uint8_t*>(ws);
#define SAKI_SCORE_ST(RK, ST)                                                                 \
  launch_score<RK, ST>(ix, B, H_q, H_kv, index_heads, N_cap, N_valid, q, q_pos, Q, B_q, mu, k, \
                       top_idx, top_score, w, p, s)
#define SAKI_SCORE(RK)                          \
  do {                                          \
    if (sketch_dtype == SAKI_FP8)               \
      SAKI_SCORE_ST(RK, kStFp8);                \
    else if (sketch_dtype == SAKI_BF16)         \
      SAKI_SCORE_ST(RK, kStBf16);               \
    else                                        \
      SAKI_SCORE_ST(RK, kStF32);                \
  } while (0)
  switch (r) {
    case 16: SAKI_SCORE(16); break;
    case 32: SAKI_SCORE(32); break;
    case 64: SAKI_SCORE(64); break;
    default: SAKI_SCORE(128); break;
  }
#undef SAKI_SCORE
#undef SAKI_SCORE_ST
  return launch_ok() ? SAKI_OK : SAKI_ERR_HIP;
}

}  // namespace

// ---------------------------------------------------------------- C ABI

extern "C" {

int saki_build_index(const void* keys, int key_dtype, int B, int H_q, int H_kv,
                     int N_cap, int d, int r, const float* B_k, const float* mu,
                     int sketch_dtype, void* index, size_t index_bytes, int n_begin,
                     int n_count, void* stream) {
  int st = check_common(B, H_q, H_kv, N_cap, 0, d);
  if (st != SAKI_OK) return st;
  if (!keys || !B_k || !mu || !index) return SAKI_ERR_ARG;
  if (!dtype_ok(key_dtype) || !sketch_ok(sketch_dtype) || !saki::rank_supported(r))
    return SAKI_ERR_UNSUPPORTED;
  if (n_begin < 0 || n_count < 0 || (long long)n_begin + n_count > N_cap) return SAKI_ERR_ARG;
  if (index_bytes < saki::index_bytes(B, H_q, N_cap, r, sketch_dtype)) return SAKI_ERR_WORKSPACE;
  if (n_count == 0) return SAKI_OK;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* ix = reinterpret_cast<uint8_t*>(index);
  const int n_end = n_begin + n_count;
#define SAKI_BUILD_ST(RK, KB)                                                                \
  do {                                                                                       \
    if (sketch_dtype == SAKI_FP8)                                                            \
      launch_build<RK, KB, kStFp8>(keys, B_k, mu, B, H_q, H_kv, N_cap, ix, n_begin, n_end, s);  \
    else if (sketch_dtype == SAKI_BF16)                                                      \
      launch_build<RK, KB, kStBf16>(keys, B_k, mu, B, H_q, H_kv, N_cap, ix, n_begin, n_end, s); \
    else                                                                                     \
      launch_build<RK, KB, kStF32>(keys, B_k, mu, B, H_q, H_kv, N_cap, ix, n_begin, n_end, s);  \
  } while (0)
#define SAKI_BUILD(RK)                         \
  do {                                         \
    if (key_dtype == SAKI_BF16)                \
      SAKI_BUILD_ST(RK, true);                 \
    else                                       \
      SAKI_BUILD_ST(RK, false);                \
  } while (0)
  switch (r) {
    case 16: SAKI_BUILD(16); break;
    case 32: SAKI_BUILD(32); break;
    case 64: SAKI_BUILD(64); break;
    default: SAKI_BUILD(128); break;
  }
#undef SAKI_BUILD
#undef SAKI_BUILD_ST
  return launch_ok() ? SAKI_OK : SAKI_ERR_HIP;
}

int saki_index_export(const void* index, int sketch_dtype, int B, int H_q, int N_cap, int r,
                      float* out, void* stream) {
  if (!index || !out || B <= 0 || H_q <= 0 || N_cap < 0) return SAKI_ERR_ARG;
  if ((long long)B * H_q > 65535) return SAKI_ERR_UNSUPPORTED;
  if (!sketch_ok(sketch_dtype) || !saki::rank_supported(r)) return SAKI_ERR_UNSUPPORTED;
  if (N_cap == 0) return SAKI_OK;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  dim3 grid((unsigned)saki::n_tiles(N_cap), B * H_q);
  const uint8_t* ix = reinterpret_cast<const uint8_t*>(index);
  const int nt = (int)saki::n_tiles(N_cap);
#define SAKI_EXPORT(RK)                                                                          \
  do {                                                                                           \
    if (sketch_dtype == SAKI_FP8)                                                                \
      hipLaunchKernelGGL((export_kernel<RK, kStFp8>), grid, dim3(64), 0, s, ix, nt, N_cap, out);   \
    else if (sketch_dtype == SAKI_BF16)                                                          \
      hipLaunchKernelGGL((export_kernel<RK, kStBf16>), grid, dim3(64), 0, s, ix, nt, N_cap, out);  \
    else                                                                                         \
      hipLaunchKernelGGL((export_kernel<RK, kStF32>), grid, dim3(64), 0, s, ix, nt, N_cap, out);   \
  } while (0)
  switch (r) {
    case 16: SAKI_EXPORT(16); break;
    case 32: SAKI_EXPORT(32); break;
    case 64: SAKI_EXPORT(64); break;
    default: SAKI_EXPORT(128); break;
  }
#undef SAKI_EXPORT
  return launch_ok() ? SAKI_OK : SAKI_ERR_HIP;
}

int saki_score_topk(const void* index, int sketch_dtype, int B, int H_q, int H_kv,
                    int index_heads, int N_cap, int N_valid, int d, int r, const float* q,
                    const int* q_pos, int Q, const float* B_q, const float* mu, int k,
                    int* top_idx, float* top_score, void* ws, size_t ws_bytes, void* stream) {
  if (!ws) return SAKI_ERR_ARG;
  return score_topk_impl(index, sketch_dtype, B, H_q, H_kv, index_heads, N_cap, N_valid, d, r,
                         q, q_pos, Q, B_q, mu, k, top_idx, top_score, ws, ws_bytes, stream);
}

int saki_score_topk_noalloc(const void* index, int sketch_dtype, int B, int H_q, int H_kv,
                            int index_heads, int N_cap, int N_valid, int d, int r,
                            const float* q, const int* q_pos, int Q, const float* B_q,
                            const float* mu, int k, int* top_idx, float* top_score,
                            void* stream) {
  return score_topk_impl(index, sketch_dtype, B, H_q, H_kv, index_heads, N_cap, N_valid, d, r,
                         q, q_pos, Q, B_q, mu, k, top_idx, top_score, nullptr, kScratchBytes,
                         stream);
}

size_t saki_noalloc_scratch_bytes(void) { return kScratchBytes; }

int saki_calibration_moments(const float* q_cal, const float* k_cal, int H_q, int H_kv,
                             int T, int d, double* Sigma_q, double* Sigma_k,
                             double* key_mean, void* stream) {
  if (!q_cal || !k_cal || !Sigma_q || !Sigma_k || !key_mean) return SAKI_ERR_ARG;
  if (H_q <= 0 || H_kv <= 0 || T <= 0 || d <= 0 || d > 4096) return SAKI_ERR_ARG;
  if ((long long)H_q + H_kv > 65535) return SAKI_ERR_UNSUPPORTED;
  const long long nb = (d + kMomBlk - 1) / kMomBlk;
  hipLaunchKernelGGL(moments_kernel, dim3((unsigned)((H_q + H_kv) * (nb * (nb + 1) / 2))), dim3(256), 0,
                     reinterpret_cast<hipStream_t>(stream), q_cal, k_cal, H_q, T, d, Sigma_q,
                     Sigma_k, key_mean);
  return launch_ok() ? SAKI_OK : SAKI_ERR_HIP;
}

int saki_recall(const void* keys, int key_dtype, const float* q, const int* q_pos, int B,
                int H_q, int H_kv, int N_cap, int N_valid, int Q, int d, int k,
                const int* approx_idx, int* hits, int* exact_idx, void* ws, size_t ws_bytes,
                void* stream) {
  int st = check_common(B, H_q, H_kv, N_cap, N_valid, d);
  if (st != SAKI_OK) return st;
  if (Q < 0) return SAKI_ERR_ARG;
  if (!dtype_ok(key_dtype) || k < 1 || k > kMaxK) return SAKI_ERR_UNSUPPORTED;
  if (Q == 0) return SAKI_OK;
  if (!keys || !q || !approx_idx || !hits) return SAKI_ERR_ARG;
  const saki::Plan p = saki::recall_plan(B, H_q, H_kv, Q, N_valid);
  if (ws_bytes < p.ws_bytes) return SAKI_ERR_WORKSPACE;
  if (p.ws_bytes > 0 && !ws) return SAKI_ERR_ARG;
  if ((size_t)p.row_blocks * p.n_chunks > 0x7fffffffu) return SAKI_ERR_UNSUPPORTED;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* w = reinterpret_cast<uint8_t*>(ws);
  if (key_dtype == SAKI_BF16)
    launch_recall<true>(keys, q, q_pos, B, H_q, H_kv, N_cap, N_valid, Q, k, approx_idx, hits,
                        exact_idx, w, p, s);
  else
    launch_recall<false>(keys, q, q_pos, B, H_q, H_kv, N_cap, N_valid, Q, k, approx_idx, hits,
                         exact_idx, w, p, s);
  return launch_ok() ? SAKI_OK : SAKI_ERR_HIP;
}

int saki_attend(const void* keys, int key_dtype, const float* values, const void* index,
                int sketch_dtype, int key_source, int B, int H_q, int H_kv, int index_heads,
                int N_cap, int N_valid, int d, int r, const float* q, const int* q_pos, int Q,
                const float* B_q, const float* mu, const int* top_idx, int k,
                float rope_theta, float* out, void* stream) {
  int st = check_common(B, H_q, H_kv, N_cap, N_valid, d);
  if (st != SAKI_OK) return st;
  if (Q < 0 || k < 1 || !(rope_theta > 0.f) || !std::isfinite(rope_theta)) return SAKI_ERR_ARG;
  if (k > kMaxK) return SAKI_ERR_UNSUPPORTED;
  const bool recon = key_source == SAKI_KEYS_RECONSTRUCTED;
  if (key_source != SAKI_KEYS_EXACT && !recon) return SAKI_ERR_ARG;
  if (Q == 0) return SAKI_OK;
  if (N_valid < 1 || !values || !q || !top_idx || !out) return SAKI_ERR_ARG;
  if (recon) {
    if (!index || !B_q || !mu) return SAKI_ERR_ARG;
    if (index_heads <= 0 || H_q % index_heads != 0 || index_heads % H_kv != 0) return SAKI_ERR_ARG;
    if (!sketch_ok(sketch_dtype) || !saki::rank_supported(r)) return SAKI_ERR_UNSUPPORTED;
  } else {
    if (!keys) return SAKI_ERR_ARG;
    if (!dtype_ok(key_dtype)) return SAKI_ERR_UNSUPPORTED;
  }
  if ((Q + kAttendWaves - 1) / kAttendWaves > 0x7fffffff) return SAKI_ERR_UNSUPPORTED;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const uint8_t* ix = reinterpret_cast<const uint8_t*>(index);
#define SAKI_ATTEND(RK, KB, ST, RC)                                                              \
  launch_attend<RK, KB, ST, RC>(keys, values, ix, B, H_q, H_kv, index_heads, N_cap, N_valid, q, \
                                q_pos, Q, B_q, mu, top_idx, k, rope_theta, out, s)
#define SAKI_ATTEND_R(RK)                              \
  do {                                                 \
    if (sketch_dtype == SAKI_FP8)                      \
      SAKI_ATTEND(RK, false, kStFp8, true);            \
    else if (sketch_dtype == SAKI_BF16)                \
      SAKI_ATTEND(RK, false, kStBf16, true);           \
    else                                               \
      SAKI_ATTEND(RK, false, kStF32, true);            \
  } while (0)
  if (!recon) {
    if (key_dtype == SAKI_BF16)
      SAKI_ATTEND(32, true, kStF32, false);
    else
      SAKI_ATTEND(32, false, kStF32, false);
  } else {
    switch (r) {
      case 16: SAKI_ATTEND_R(16); break;
      case 32: SAKI_ATTEND_R(32); break;
      case 64: SAKI_ATTEND_R(64); break;
      default: SAKI_ATTEND_R(128); break;
    }
  }
#undef SAKI_ATTEND_R
#undef SAKI_ATTEND
  return launch_ok() ? SAKI_OK : SAKI_ERR_HIP;
}

}  // extern "C"
