// Wave-level running top-64 selection for gfx950 (wave64).  Device code,
// included by saki_kernels.hip only.
//
// Ranking: score descending, then key index ascending (ties go to the lower
// index).  Both orders are folded into one integer key so that every
// compare-exchange is a single unsigned comparison, with no branches:
//   float scores : 64-bit key  = ordered(score bits) << 32 | ~index
//   double scores: (64-bit ordered score bits, 32-bit ~index) compared
//                  lexicographically
// where ordered() maps IEEE bits to an unsigned integer of the same order.
//
// A row's list holds its 64 best keys, one per lane, sorted (lane 0 best).
// Candidates are filtered against the list's 64th score; the few that pass
// are appended to a per-row LDS buffer, and when the buffer is full the wave
// sorts it with a bitonic network and merges it into the list (lane i takes
// max(A_i, B_{63-i}), then a bitonic half-cleaner cascade).  Each wave visits
// its keys in increasing index order, so a candidate whose score only equals
// the 64th score can never outrank it: the strict filter `score > threshold`
// is exact.
#pragma once

#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstdint>

namespace saki_dev {

constexpr int kWave = 64;
constexpr int kList = 64;  // list length == wave size
constexpr int kPadIdx = INT_MAX;

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }

__device__ __forceinline__ int prefix_count(uint64_t mask) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// Orders the LDS accesses of one wave: writes by some lanes become visible to
// reads by other lanes of the same wave issued after this point.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ uint32_t readlane_u32(uint32_t v, int l) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, l);
}
__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int l) {
  return ((uint64_t)readlane_u32((uint32_t)(v >> 32), l) << 32) | readlane_u32((uint32_t)v, l);
}
__device__ __forceinline__ float readlane_s(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ __forceinline__ double readlane_s(double v, int l) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  return __longlong_as_double((long long)readlane_u64(u, l));
}

// ---------------------------------------------------------------- lane shuffles

// v from lane (lane ^ m), m a power of two below 64, on the VALU only: DPP
// quad permutes (m = 1, 2), DPP row rotations (m = 4, 8) and the gfx950
// permlane swaps (m = 16, 32).  m must fold to a constant after unrolling.
__device__ __forceinline__ uint32_t xor_shfl_u32(uint32_t v, int m) {
  const int x = (int)v;
  switch (m) {
    case 1: return (uint32_t)__builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, false);
    case 2: return (uint32_t)__builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, false);
    case 4: {
      const int up = __builtin_amdgcn_mov_dpp(x, 0x12C, 0xF, 0xF, false);  // lane+4 (mod 16)
      const int dn = __builtin_amdgcn_mov_dpp(x, 0x124, 0xF, 0xF, false);  // lane-4 (mod 16)
      return (uint32_t)((lane_id() & 4) ? dn : up);
    }
    case 8: return (uint32_t)__builtin_amdgcn_mov_dpp(x, 0x128, 0xF, 0xF, false);
    case 16: {
      const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
      return (lane_id() & 16) ? r[0] : r[1];
    }
    default: {
      const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
      return (lane_id() & 32) ? r[0] : r[1];
    }
  }
}
// v from lane 63 - lane: mirror within rows of 16, then swap the rows.
__device__ __forceinline__ uint32_t rev_shfl_u32(uint32_t v) {
  const uint32_t m = (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x140, 0xF, 0xF, false);
  return xor_shfl_u32(xor_shfl_u32(m, 16), 32);
}
__device__ __forceinline__ uint64_t xor_shfl_u64(uint64_t v, int m) {
  return ((uint64_t)xor_shfl_u32((uint32_t)(v >> 32), m) << 32) | xor_shfl_u32((uint32_t)v, m);
}
__device__ __forceinline__ uint64_t rev_shfl_u64(uint64_t v) {
  return ((uint64_t)rev_shfl_u32((uint32_t)(v >> 32)) << 32) | rev_shfl_u32((uint32_t)v);
}

// ---------------------------------------------------------------- ordered keys

__device__ __forceinline__ uint32_t ord_f32(float s) {
  const uint32_t u = __float_as_uint(s);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float unord_f32(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}
__device__ __forceinline__ uint64_t ord_f64(double s) {
  const uint64_t u = (uint64_t)__double_as_longlong(s);
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}
__device__ __forceinline__ double unord_f64(uint64_t o) {
  return __longlong_as_double((long long)((o >> 63) ? (o & 0x7fffffffffffffffull) : ~o));
}

// Key operations for float scores: one 64-bit integer per entry.
struct KeysF32 {
  using K = uint64_t;
  using S = float;
  __device__ static K make(float s, int j) {
    return ((uint64_t)ord_f32(s) << 32) | (uint32_t)(~(uint32_t)j);
  }
  __device__ static K pad() { return make(-INFINITY, kPadIdx); }
  __device__ static bool gt(K a, K b) { return a > b; }
  __device__ static K sel(bool c, K a, K b) { return c ? a : b; }
  __device__ static K shfl_xor(K a, int m) { return xor_shfl_u64(a, m); }
  __device__ static K reverse(K a) { return rev_shfl_u64(a); }
  __device__ static K readlane(K a, int l) { return readlane_u64(a, l); }
  __device__ static float score(K a) { return unord_f32((uint32_t)(a >> 32)); }
  __device__ static int index(K a) { return (int)~(uint32_t)a; }
};

// Plain 32-bit unsigned keys (the caller packs whatever order it needs).
struct KeysU32 {
  using K = uint32_t;
  __device__ static bool gt(K a, K b) { return a > b; }
  __device__ static K sel(bool c, K a, K b) { return c ? a : b; }
  __device__ static K shfl_xor(K a, int m) { return xor_shfl_u32(a, m); }
  __device__ static K reverse(K a) { return rev_shfl_u32(a); }
};

// Key operations for double scores: (ordered bits, ~index).
struct KeyF64 {
  uint64_t s;
  uint32_t j;
};
struct KeysF64 {
  using K = KeyF64;
  using S = double;
  __device__ static K make(double s, int j) { return {ord_f64(s), ~(uint32_t)j}; }
  __device__ static K pad() { return make(-(double)INFINITY, kPadIdx); }
  __device__ static bool gt(K a, K b) { return (a.s > b.s) | ((a.s == b.s) & (a.j > b.j)); }
  __device__ static K sel(bool c, K a, K b) {
    K r;
    r.s = c ? a.s : b.s;
    r.j = c ? a.j : b.j;
    return r;
  }
  __device__ static K shfl_xor(K a, int m) { return {xor_shfl_u64(a.s, m), xor_shfl_u32(a.j, m)}; }
  __device__ static K reverse(K a) { return {rev_shfl_u64(a.s), rev_shfl_u32(a.j)}; }
  __device__ static K readlane(K a, int l) { return {readlane_u64(a.s, l), readlane_u32(a.j, l)}; }
  __device__ static double score(K a) { return unord_f64(a.s); }
  __device__ static int index(K a) { return (int)~a.j; }
};

// ---------------------------------------------------------------- wave networks

// Bitonic sort of one key per lane into descending order (lane 0 best).
template <class KO>
__device__ __forceinline__ void wave_sort(typename KO::K& x) {
  const int lane = lane_id();
#pragma unroll
  for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
    for (int m = k >> 1; m > 0; m >>= 1) {
      const typename KO::K o = KO::shfl_xor(x, m);
      const bool want_better = ((lane & k) == 0) == ((lane & m) == 0);
      const bool mine = KO::gt(x, o);
      x = KO::sel(want_better == mine, x, o);
    }
  }
}

// a <- the 64 best of (a U b), sorted; both inputs sorted descending.
template <class KO>
__device__ __forceinline__ void wave_merge(typename KO::K& a, typename KO::K b) {
  const int lane = lane_id();
  const typename KO::K r = KO::reverse(b);
  a = KO::sel(KO::gt(r, a), r, a);
#pragma unroll
  for (int m = kWave / 2; m > 0; m >>= 1) {
    const typename KO::K o = KO::shfl_xor(a, m);
    const bool low = (lane & m) == 0;
    a = KO::sel(low == KO::gt(a, o), a, o);
  }
}

// ---------------------------------------------------------------- per-row lists

// Running top-64 lists of R rows owned by one wave.  Lists and candidate
// buffers live in LDS (so the row index may be a run-time value); the
// threshold score and buffer count of row r are held by lane r of two
// registers.  Buffers have 64 slots and are flushed before a batch of
// candidates would overflow them.
template <class KO, int R>
struct RowLists {
  using K = typename KO::K;
  using S = typename KO::S;
  K* list;  // LDS [R][64]
  K* buf;   // LDS [R][64]
  S thr;    // lane r: 64th score of row r (-inf while the list is not full)
  int cnt;  // lane r: buffered candidates of row r

  __device__ void init(K* list_mem, K* buf_mem) {
    list = list_mem;
    buf = buf_mem;
    const int lane = lane_id();
    for (int r = 0; r < R; ++r) list[r * kList + lane] = KO::pad();
    thr = -(S)INFINITY;
    cnt = 0;
    wave_lds_sync();
  }

  __device__ __forceinline__ S threshold(int r) const { return readlane_s(thr, r); }
  __device__ __forceinline__ int count(int r) const { return __builtin_amdgcn_readlane(cnt, r); }

  // Sort row r's buffer and merge it into the list.
  __device__ void flush(int r) {
    const int lane = lane_id();
    const int c = count(r);
    wave_lds_sync();
    K b = lane < c ? buf[r * kList + lane] : KO::pad();
    wave_sort<KO>(b);
    K a = list[r * kList + lane];
    wave_merge<KO>(a, b);
    list[r * kList + lane] = a;
    const S t = KO::score(KO::readlane(a, kWave - 1));
    if (lane == r) { thr = t; cnt = 0; }
    wave_lds_sync();
  }

  // One candidate score per lane for row r (masked lanes pass -inf).
  __device__ __forceinline__ void offer(int r, S s, int j) {
    const S t = threshold(r);
    bool take = s > t;
    uint64_t mask = __ballot(take);
    if (mask == 0) return;
    int c = count(r);
    if (c + __popcll(mask) > kList) {
      flush(r);
      take = s > threshold(r);
      mask = __ballot(take);
      if (mask == 0) return;
      c = 0;
    }
    if (take) buf[r * kList + c + prefix_count(mask)] = KO::make(s, j);
    c += __popcll(mask);
    if (lane_id() == r) cnt = c;
    if (c == kList) flush(r);
  }

  __device__ void finish(int r) {
    if (count(r) > 0) flush(r);
  }

  // Row r's final entry for this lane (lane 0 = best).
  __device__ K entry(int r) const { return list[r * kList + lane_id()]; }
};

}  // namespace saki_dev
