// GPU side of libsaki for gfx950 (CDNA4, wave64).
//
// Kernels (one launch each, all on the caller's stream):
//   build_index_kernel   key codes c = B_k^T (k - mu) for every query head (Eq. 4)
//   query_sketch_kernel  z = B_q^T q and b = q^T mu per query row (Sec. 6)
//   score_topk_kernel    s = z . c + b over a row's visible keys, running top-64
//   exact_topk_kernel    exact float64 q . k, running top-64, recall hits (Sec. 3)
//   merge_kernel         reduces per-chunk partial top-64 lists of one row
//   export_kernel        debug read-back of the codes
//
// Top-k selection.  A row's running top-64 lives in one wave, one entry per
// lane, sorted by (score desc, index asc).  New candidates are compared with
// the current 64th entry; the few that beat it are appended to a per-row LDS
// buffer, and when 64 have gathered the wave sorts them with a bitonic network
// and merges them into the list (max(A_i, B_{63-i}) followed by a bitonic
// merge).  Each wave visits its keys in increasing index order, so a
// candidate that only ties the threshold's score can never outrank it.

#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstdint>

#include "saki.h"
#include "saki_internal.h"

namespace {

using saki::kMaxK;
using saki::kTile;

constexpr int kWave = 64;
constexpr int kMaxWaves = 4;
constexpr int kBuf = 128;  // candidate buffer slots per row
constexpr int kPadIdx = INT_MAX;

// ---------------------------------------------------------------- helpers

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }

__device__ __forceinline__ int prefix_count(uint64_t mask) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// Orders LDS accesses of one wave: writes by some lanes become visible to
// reads by other lanes issued after this point.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ float bcast(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ __forceinline__ int bcast(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ __forceinline__ double bcast(double v, int l) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

template <class S>
__device__ __forceinline__ S neg_inf() { return -INFINITY; }

// Strict ranking order: a before b.
template <class S>
__device__ __forceinline__ bool better(S as, int aj, S bs, int bj) {
  return as > bs || (as == bs && aj < bj);
}

// Bitonic sort of one entry per lane into descending rank order.
template <class S>
__device__ __forceinline__ void wave_sort(S& s, int& j) {
  const int lane = lane_id();
#pragma unroll
  for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
    for (int m = k >> 1; m > 0; m >>= 1) {
      const S os = __shfl_xor(s, m, kWave);
      const int oj = __shfl_xor(j, m, kWave);
      const bool desc = (lane & k) == 0;
      const bool low = (lane & m) == 0;
      const bool mine = better(s, j, os, oj);
      const bool keep = (low == desc) ? mine : !mine;
      if (!keep) { s = os; j = oj; }
    }
  }
}

// list <- top 64 of (list U b), both sorted descending.
template <class S>
__device__ __forceinline__ void wave_merge(S& ls, int& lj, S bs, int bj) {
  const int lane = lane_id();
  const S rs = __shfl(bs, kWave - 1 - lane, kWave);
  const int rj = __shfl(bj, kWave - 1 - lane, kWave);
  if (better(rs, rj, ls, lj)) { ls = rs; lj = rj; }
#pragma unroll
  for (int m = kWave / 2; m > 0; m >>= 1) {
    const S os = __shfl_xor(ls, m, kWave);
    const int oj = __shfl_xor(lj, m, kWave);
    const bool low = (lane & m) == 0;
    const bool mine = better(ls, lj, os, oj);
    const bool keep = low ? mine : !mine;
    if (!keep) { ls = os; lj = oj; }
  }
}

// Running top-64 of R rows owned by one wave.
template <class S, int R>
struct WaveTopK {
  S ls[R];
  int lj[R];
  S ts[R];    // current 64th score (wave-uniform)
  int tj[R];  // and its index
  int cnt[R]; // buffered candidates (wave-uniform)
  S* bs;      // LDS [R][kBuf]
  int* bj;

  __device__ void init(S* sbuf, int* jbuf) {
    bs = sbuf;
    bj = jbuf;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      ls[r] = neg_inf<S>();
      lj[r] = kPadIdx;
      ts[r] = neg_inf<S>();
      tj[r] = kPadIdx;
      cnt[r] = 0;
    }
  }

  __device__ void flush(int r) {
    const int lane = lane_id();
    wave_lds_sync();
    S s = bs[r * kBuf + lane];
    int j = bj[r * kBuf + lane];
    if (lane >= cnt[r]) { s = neg_inf<S>(); j = kPadIdx; }
    wave_sort(s, j);
    wave_merge(ls[r], lj[r], s, j);
    ts[r] = bcast(ls[r], kWave - 1);
    tj[r] = bcast(lj[r], kWave - 1);
    const int rem = cnt[r] - kWave;
    if (rem > 0 && lane < rem) {
      const S s2 = bs[r * kBuf + kWave + lane];
      const int j2 = bj[r * kBuf + kWave + lane];
      bs[r * kBuf + lane] = s2;
      bj[r * kBuf + lane] = j2;
    }
    cnt[r] = rem > 0 ? rem : 0;
    wave_lds_sync();
  }

  // One candidate per lane for row r.
  __device__ __forceinline__ void offer(int r, S s, int j) {
    const bool take = better(s, j, ts[r], tj[r]);
    const uint64_t mask = __ballot(take);
    if (mask == 0) return;
    const int pos = cnt[r] + prefix_count(mask);
    if (take) {
      bs[r * kBuf + pos] = s;
      bj[r * kBuf + pos] = j;
    }
    cnt[r] += __popcll(mask);
    if (cnt[r] >= kWave) flush(r);
  }

  __device__ void finish(int r) {
    if (cnt[r] > 0) flush(r);
  }
};

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t bf16_bits(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}
__device__ __forceinline__ float bf16_round(float x) { return __uint_as_float(bf16_bits(x) << 16); }

template <bool BF>
__device__ __forceinline__ float load_key_elem(const void* p, size_t i) {
  if constexpr (BF) {
    const uint16_t v = reinterpret_cast<const uint16_t*>(p)[i];
    return __uint_as_float((uint32_t)v << 16);
  } else {
    return reinterpret_cast<const float*>(p)[i];
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

// ---------------------------------------------------------------- build index

// grid (tiles, H_q, B), block 256.  One tile of 64 keys per workgroup.
template <int RK, bool KBF, bool SBF>
__global__ __launch_bounds__(256) void build_index_kernel(
    const void* __restrict__ keys, const float* __restrict__ Bk,
    const float* __restrict__ mu, int H_q, int H_kv, int N_cap, int n_tiles,
    uint8_t* __restrict__ index, int n_begin, int n_end, int tile0) {
  constexpr int D = saki::kHeadDim;
  constexpr int ES = SBF ? 2 : 4;
  constexpr int CPP = saki::kChunkBytes / ES;  // code elements per piece
  constexpr int NP = RK / CPP;                 // pieces per key
  __shared__ float ks[kTile][D + 1];
  __shared__ float bk[D][RK];
  const int tile = tile0 + blockIdx.x;
  const int h = blockIdx.y, b = blockIdx.z;
  const int g = h / (H_q / H_kv);
  const int tid = threadIdx.x;
  const size_t key_base = ((size_t)b * H_kv + g) * N_cap;
  for (int i = tid; i < kTile * D; i += 256) {
    const int t = i / D, c = i % D;
    const int n = tile * kTile + t;
    float v = 0.f;
    if (n < N_cap) v = load_key_elem<KBF>(keys, (key_base + n) * D + c) - mu[(size_t)g * D + c];
    ks[t][c] = v;
  }
  for (int i = tid; i < D * RK; i += 256) bk[i / RK][i % RK] = Bk[(size_t)h * D * RK + i];
  __syncthreads();
  uint8_t* tbase = index + (((size_t)b * H_q + h) * n_tiles + tile) * ((size_t)kTile * RK * (SBF ? 2 : 4));
  for (int p = tid; p < kTile * NP; p += 256) {
    const int t = p % kTile, piece = p / kTile;
    const int n = tile * kTile + t;
    float acc[CPP];
#pragma unroll
    for (int e = 0; e < CPP; ++e) acc[e] = 0.f;
    for (int c = 0; c < D; ++c) {
      const float kv = ks[t][c];
#pragma unroll
      for (int e = 0; e < CPP; ++e) acc[e] = fmaf(kv, bk[c][piece * CPP + e], acc[e]);
    }
    if (n >= n_begin && n < n_end) {
      uint4 out;
      if constexpr (SBF) {
        out.x = bf16_bits(acc[0]) | (bf16_bits(acc[1]) << 16);
        out.y = bf16_bits(acc[2]) | (bf16_bits(acc[3]) << 16);
        out.z = bf16_bits(acc[4]) | (bf16_bits(acc[5]) << 16);
        out.w = bf16_bits(acc[6]) | (bf16_bits(acc[7]) << 16);
      } else {
        out.x = __float_as_uint(acc[0]);
        out.y = __float_as_uint(acc[1]);
        out.z = __float_as_uint(acc[2]);
        out.w = __float_as_uint(acc[3]);
      }
      *reinterpret_cast<uint4*>(tbase + (size_t)piece * kTile * 16 + (size_t)t * 16) = out;
    }
  }
}

// grid (tiles, B*H_q), block 64: codes -> float [B, H_q, N_cap, r].
template <int RK, bool SBF>
__global__ __launch_bounds__(64) void export_kernel(const uint8_t* __restrict__ index,
                                                    int n_tiles, int N_cap,
                                                    float* __restrict__ out) {
  constexpr int ES = SBF ? 2 : 4;
  constexpr int CPP = saki::kChunkBytes / ES;
  constexpr int NP = RK / CPP;
  const int tile = blockIdx.x;
  const size_t bh = blockIdx.y;
  const int t = threadIdx.x;
  const int n = tile * kTile + t;
  if (n >= N_cap) return;
  const uint8_t* tbase = index + (bh * n_tiles + tile) * ((size_t)kTile * RK * (SBF ? 2 : 4));
  for (int piece = 0; piece < NP; ++piece) {
    const uint4 v = *reinterpret_cast<const uint4*>(tbase + (size_t)piece * kTile * 16 + (size_t)t * 16);
    float f[CPP];
    unpack_piece<SBF>(v, f);
    for (int e = 0; e < CPP; ++e) out[(bh * N_cap + n) * RK + piece * CPP + e] = f[e];
  }
}

// ---------------------------------------------------------------- query sketch

// grid (ceil(Q/16), B*H_q), block 256.  z = B_q^T q (float32, rounded to bf16
// when the sketches are bf16), b = q^T mu.
template <int RK, bool SBF>
__global__ __launch_bounds__(256) void query_sketch_kernel(
    const float* __restrict__ q, const float* __restrict__ Bq,
    const float* __restrict__ mu, int H_q, int H_kv, int Q, float* __restrict__ z,
    float* __restrict__ bout) {
  constexpr int D = saki::kHeadDim;
  constexpr int QR = 16;
  __shared__ float bq[D][RK];
  __shared__ float qs[QR][D];
  __shared__ float ms[D];
  const int bh = blockIdx.y;
  const int h = bh % H_q;
  const int g = h / (H_q / H_kv);
  const int i0 = blockIdx.x * QR;
  const int tid = threadIdx.x;
  for (int i = tid; i < D * RK; i += 256) bq[i / RK][i % RK] = Bq[(size_t)h * D * RK + i];
  for (int i = tid; i < QR * D; i += 256) {
    const int rr = i / D;
    qs[rr][i % D] = (i0 + rr < Q) ? q[((size_t)bh * Q + i0 + rr) * D + (i % D)] : 0.f;
  }
  if (tid < D) ms[tid] = mu[(size_t)g * D + tid];
  __syncthreads();
  for (int o = tid; o < QR * (RK + 1); o += 256) {
    const int rr = o / (RK + 1), m = o % (RK + 1);
    const int i = i0 + rr;
    if (i >= Q) continue;
    float acc = 0.f;
    if (m < RK) {
      for (int c = 0; c < D; ++c) acc = fmaf(qs[rr][c], bq[c][m], acc);
      if (SBF) acc = bf16_round(acc);
      z[((size_t)bh * Q + i) * RK + m] = acc;
    } else {
      for (int c = 0; c < D; ++c) acc = fmaf(qs[rr][c], ms[c], acc);
      bout[(size_t)bh * Q + i] = acc;
    }
  }
}

__device__ __forceinline__ int row_limit(int i, int Q, int N_valid, const int* q_pos) {
  if (i >= Q) return 0;
  if (!q_pos) return N_valid;
  const long long lim = (long long)q_pos[i] + 1;
  return lim < 0 ? 0 : (lim > N_valid ? N_valid : (int)lim);
}

// ---------------------------------------------------------------- sketch scoring

// grid (row_blocks * n_chunks, B*H_q), block 64*waves.  Each wave owns R rows.
template <int RK, bool SBF, int R>
__global__ __launch_bounds__(256) void score_topk_kernel(
    const uint8_t* __restrict__ index, int n_tiles, int N_valid, int Q,
    const int* __restrict__ q_pos, const float* __restrict__ z,
    const float* __restrict__ bvec, int row_blocks, int chunk, int n_chunks, int k,
    int* __restrict__ top_idx, float* __restrict__ top_score,
    float* __restrict__ part_s, int* __restrict__ part_j) {
  constexpr int ES = SBF ? 2 : 4;
  constexpr int CPP = saki::kChunkBytes / ES;
  constexpr int NP = RK / CPP;
  __shared__ float zs[kMaxWaves][R][RK];
  __shared__ float sbuf[kMaxWaves][R][kBuf];
  __shared__ int jbuf[kMaxWaves][R][kBuf];
  const int wave = threadIdx.x / kWave, lane = lane_id();
  const int waves = blockDim.x / kWave;
  const int rb = blockIdx.x % row_blocks, ch = blockIdx.x / row_blocks;
  const size_t bh = blockIdx.y;
  const int row0 = (rb * waves + wave) * R;
  if (row0 >= Q) return;

  int lim[R];
  float bb[R];
  int kmax = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    lim[r] = row_limit(row0 + r, Q, N_valid, q_pos);
    kmax = lim[r] > kmax ? lim[r] : kmax;
    bb[r] = (row0 + r < Q) ? bvec[bh * Q + row0 + r] : 0.f;
  }
  for (int i = lane; i < R * RK; i += kWave) {
    const int r = i / RK;
    zs[wave][r][i % RK] = (row0 + r < Q) ? z[(bh * Q + row0 + r) * RK + (i % RK)] : 0.f;
  }
  wave_lds_sync();

  WaveTopK<float, R> top;
  top.init(&sbuf[wave][0][0], &jbuf[wave][0][0]);
  const int kbeg = ch * chunk;
  const int kend = min(kbeg + chunk, kmax);
  const uint8_t* hbase = index + bh * n_tiles * ((size_t)kTile * RK * (SBF ? 2 : 4));
  for (int t0 = kbeg; t0 < kend; t0 += kTile) {
    const int j = t0 + lane;
    const uint8_t* tb = hbase + (size_t)(t0 / kTile) * ((size_t)kTile * RK * (SBF ? 2 : 4));
    float c[RK];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const uint4 v = *reinterpret_cast<const uint4*>(tb + (size_t)p * kTile * 16 + (size_t)lane * 16);
      unpack_piece<SBF>(v, c + p * CPP);
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      float acc = 0.f;
#pragma unroll
      for (int m = 0; m < RK; ++m) acc = fmaf(zs[wave][r][m], c[m], acc);
      const bool ok = j < lim[r];
      top.offer(r, ok ? acc + bb[r] : -INFINITY, ok ? j : kPadIdx);
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    top.finish(r);
    const int i = row0 + r;
    if (i >= Q) continue;
    if (n_chunks == 1) {
      if (lane < k) {
        const size_t o = (bh * Q + i) * k + lane;
        top_idx[o] = top.lj[r] == kPadIdx ? -1 : top.lj[r];
        if (top_score) top_score[o] = top.ls[r];
      }
    } else {
      const size_t o = ((bh * Q + i) * n_chunks + ch) * kMaxK + lane;
      part_s[o] = top.ls[r];
      part_j[o] = top.lj[r];
    }
  }
}

// ---------------------------------------------------------------- exact scores + recall

// Hits of the exact list (one entry per lane, the first k lanes count)
// against approx_idx row `row` (length k).
__device__ __forceinline__ int row_hits(int ej, const int* __restrict__ approx, size_t row, int k) {
  const int lane = lane_id();
  const int aj = lane < k ? approx[row * k + lane] : -1;
  bool found = false;
  for (int m = 0; m < k; ++m) {
    const int v = __shfl(aj, m, kWave);
    found |= (v >= 0 && v == ej);
  }
  const bool counts = lane < k && ej != kPadIdx && found;
  return __popcll(__ballot(counts));
}

// grid (row_blocks * n_chunks, B*H_q), block 64*waves.  Exact float64 scores.
template <bool KBF, int R>
__global__ __launch_bounds__(256) void exact_topk_kernel(
    const void* __restrict__ keys, const float* __restrict__ q,
    const int* __restrict__ q_pos, int H_q, int H_kv, int N_cap, int N_valid, int Q,
    int row_blocks, int chunk, int n_chunks, int k, const int* __restrict__ approx,
    int* __restrict__ hits, int* __restrict__ exact_idx, double* __restrict__ part_s,
    int* __restrict__ part_j) {
  constexpr int D = saki::kHeadDim;
  __shared__ float qsh[kMaxWaves][R][D];
  __shared__ double sbuf[kMaxWaves][R][kBuf];
  __shared__ int jbuf[kMaxWaves][R][kBuf];
  const int wave = threadIdx.x / kWave, lane = lane_id();
  const int waves = blockDim.x / kWave;
  const int rb = blockIdx.x % row_blocks, ch = blockIdx.x / row_blocks;
  const size_t bh = blockIdx.y;
  const int b = (int)(bh / H_q), h = (int)(bh % H_q);
  const int g = h / (H_q / H_kv);
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
    qsh[wave][r][i % D] = (row0 + r < Q) ? q[(bh * Q + row0 + r) * D + (i % D)] : 0.f;
  }
  wave_lds_sync();
  WaveTopK<double, R> top;
  top.init(&sbuf[wave][0][0], &jbuf[wave][0][0]);
  const size_t kbase = ((size_t)b * H_kv + g) * N_cap;
  const int kbeg = ch * chunk;
  const int kend = min(kbeg + chunk, kmax);
  for (int t0 = kbeg; t0 < kend; t0 += kTile) {
    const int j = t0 + lane;
    const bool inb = j < N_valid;
    double acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.0;
    for (int c0 = 0; c0 < D; c0 += 8) {
      float kv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) kv[e] = inb ? load_key_elem<KBF>(keys, (kbase + j) * D + c0 + e) : 0.f;
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[r] = fma((double)qsh[wave][r][c0 + e], (double)kv[e], acc[r]);
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const bool ok = j < lim[r];
      top.offer(r, ok ? acc[r] : -(double)INFINITY, ok ? j : kPadIdx);
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    top.finish(r);
    const int i = row0 + r;
    if (i >= Q) continue;
    const size_t row = bh * Q + i;
    if (n_chunks == 1) {
      if (exact_idx && lane < k) exact_idx[row * k + lane] = top.lj[r] == kPadIdx ? -1 : top.lj[r];
      const int hsum = row_hits(top.lj[r], approx, row, k);
      if (lane == 0) hits[row] = hsum;
    } else {
      const size_t o = (row * n_chunks + ch) * kMaxK + lane;
      part_s[o] = top.ls[r];
      part_j[o] = top.lj[r];
    }
  }
}

// ---------------------------------------------------------------- merge of partials

// grid (ceil(rows/4)), block 256: one wave per row merges n_chunks sorted lists.
template <class S, bool RECALL>
__global__ __launch_bounds__(256) void merge_kernel(
    const S* __restrict__ part_s, const int* __restrict__ part_j, size_t rows,
    int n_chunks, int k, int* __restrict__ out_idx, float* __restrict__ out_score,
    const int* __restrict__ approx, int* __restrict__ hits) {
  const int lane = lane_id();
  const size_t row = (size_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
  if (row >= rows) return;
  S ls = neg_inf<S>();
  int lj = kPadIdx;
  for (int c = 0; c < n_chunks; ++c) {
    const size_t o = (row * n_chunks + c) * kMaxK + lane;
    const S s = part_s[o];
    const int j = part_j[o];
    // the partial is sorted: skip it when its best cannot enter the list
    const S s0 = bcast(s, 0);
    const int j0 = bcast(j, 0);
    const S t = bcast(ls, kWave - 1);
    const int tjx = bcast(lj, kWave - 1);
    if (!better(s0, j0, t, tjx)) continue;
    wave_merge(ls, lj, s, j);
  }
  if constexpr (RECALL) {
    if (out_idx && lane < k) out_idx[row * k + lane] = lj == kPadIdx ? -1 : lj;
    const int hsum = row_hits(lj, approx, row, k);
    if (lane == 0) hits[row] = hsum;
  } else {
    if (lane < k) {
      out_idx[row * k + lane] = lj == kPadIdx ? -1 : lj;
      if (out_score) out_score[row * k + lane] = (float)ls;
    }
  }
}

// ---------------------------------------------------------------- dispatch helpers

bool launch_ok() { return hipGetLastError() == hipSuccess; }

template <int RK, bool KBF, bool SBF>
void launch_build(const void* keys, const float* Bk, const float* mu, int B, int H_q,
                  int H_kv, int N_cap, uint8_t* index, int n_begin, int n_end,
                  hipStream_t s) {
  const int t0 = n_begin / kTile;
  const int t1 = (n_end + kTile - 1) / kTile;
  dim3 grid(t1 - t0, H_q, B);
  hipLaunchKernelGGL((build_index_kernel<RK, KBF, SBF>), grid, dim3(256), 0, s, keys, Bk,
                     mu, H_q, H_kv, N_cap, (int)saki::n_tiles(N_cap), index, n_begin,
                     n_end, t0);
}

template <int RK, bool SBF>
void launch_score(const uint8_t* index, int B, int H_q, int H_kv, int N_cap, int N_valid,
                  const float* q, const int* q_pos, int Q, const float* Bq, const float* mu,
                  int k, int* top_idx, float* top_score, uint8_t* ws,
                  const saki::Plan& p, hipStream_t s) {
  float* z = reinterpret_cast<float*>(ws + p.z_off);
  float* bv = reinterpret_cast<float*>(ws + p.b_off);
  hipLaunchKernelGGL((query_sketch_kernel<RK, SBF>), dim3((Q + 15) / 16, B * H_q),
                     dim3(256), 0, s, q, Bq, mu, H_q, H_kv, Q, z, bv);
  float* ps = nullptr;
  int* pj = nullptr;
  const size_t rows = (size_t)B * H_q * Q;
  if (p.n_chunks > 1) {
    ps = reinterpret_cast<float*>(ws + p.part_off);
    pj = reinterpret_cast<int*>(ws + p.part_off + rows * p.n_chunks * kMaxK * sizeof(float));
  }
  dim3 grid((unsigned)(p.row_blocks * p.n_chunks), B * H_q);
  const int nt = (int)saki::n_tiles(N_cap);
  if (p.rows == 4)
    hipLaunchKernelGGL((score_topk_kernel<RK, SBF, 4>), grid, dim3(kWave * p.waves), 0, s,
                       index, nt, N_valid, Q, q_pos, z, bv, p.row_blocks, p.chunk,
                       p.n_chunks, k, top_idx, top_score, ps, pj);
  else
    hipLaunchKernelGGL((score_topk_kernel<RK, SBF, 1>), grid, dim3(kWave * p.waves), 0, s,
                       index, nt, N_valid, Q, q_pos, z, bv, p.row_blocks, p.chunk,
                       p.n_chunks, k, top_idx, top_score, ps, pj);
  if (p.n_chunks > 1)
    hipLaunchKernelGGL((merge_kernel<float, false>), dim3((unsigned)((rows + 3) / 4)),
                       dim3(256), 0, s, ps, pj, rows, p.n_chunks, k, top_idx, top_score,
                       nullptr, nullptr);
}

template <bool KBF>
void launch_recall(const void* keys, const float* q, const int* q_pos, int B, int H_q,
                   int H_kv, int N_cap, int N_valid, int Q, int k, const int* approx,
                   int* hits, int* exact_idx, uint8_t* ws, const saki::Plan& p,
                   hipStream_t s) {
  double* ps = nullptr;
  int* pj = nullptr;
  const size_t rows = (size_t)B * H_q * Q;
  if (p.n_chunks > 1) {
    ps = reinterpret_cast<double*>(ws + p.part_off);
    pj = reinterpret_cast<int*>(ws + p.part_off + rows * p.n_chunks * kMaxK * sizeof(double));
  }
  dim3 grid((unsigned)(p.row_blocks * p.n_chunks), B * H_q);
  if (p.rows == 4)
    hipLaunchKernelGGL((exact_topk_kernel<KBF, 4>), grid, dim3(kWave * p.waves), 0, s, keys,
                       q, q_pos, H_q, H_kv, N_cap, N_valid, Q, p.row_blocks, p.chunk,
                       p.n_chunks, k, approx, hits, exact_idx, ps, pj);
  else
    hipLaunchKernelGGL((exact_topk_kernel<KBF, 1>), grid, dim3(kWave * p.waves), 0, s, keys,
                       q, q_pos, H_q, H_kv, N_cap, N_valid, Q, p.row_blocks, p.chunk,
                       p.n_chunks, k, approx, hits, exact_idx, ps, pj);
  if (p.n_chunks > 1)
    hipLaunchKernelGGL((merge_kernel<double, true>), dim3((unsigned)((rows + 3) / 4)),
                       dim3(256), 0, s, ps, pj, rows, p.n_chunks, k, exact_idx, nullptr,
                       approx, hits);
}

bool dtype_ok(int t) { return t == SAKI_F32 || t == SAKI_BF16; }

// Common size validation of the GPU entry points.
int check_common(int B, int H_q, int H_kv, int N_cap, int N_valid, int d) {
  if (B <= 0 || H_q <= 0 || H_kv <= 0 || H_q % H_kv != 0 || N_cap < 0 || N_valid < 0 ||
      N_valid > N_cap || d <= 0)
    return SAKI_ERR_ARG;
  if (B > 65535 || (long long)B * H_q > 65535) return SAKI_ERR_UNSUPPORTED;
  if (d != saki::kHeadDim) return SAKI_ERR_UNSUPPORTED;
  return SAKI_OK;
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
  if (!dtype_ok(key_dtype) || !dtype_ok(sketch_dtype) || !saki::rank_supported(r))
    return SAKI_ERR_UNSUPPORTED;
  if (n_begin < 0 || n_count < 0 || (long long)n_begin + n_count > N_cap) return SAKI_ERR_ARG;
  if (index_bytes < saki::index_bytes(B, H_q, N_cap, r, sketch_dtype)) return SAKI_ERR_WORKSPACE;
  if (n_count == 0) return SAKI_OK;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* ix = reinterpret_cast<uint8_t*>(index);
  const int n_end = n_begin + n_count;
#define SAKI_BUILD(RK)                                                                   \
  do {                                                                                   \
    if (key_dtype == SAKI_BF16) {                                                        \
      if (sketch_dtype == SAKI_BF16)                                                     \
        launch_build<RK, true, true>(keys, B_k, mu, B, H_q, H_kv, N_cap, ix, n_begin, n_end, s); \
      else                                                                               \
        launch_build<RK, true, false>(keys, B_k, mu, B, H_q, H_kv, N_cap, ix, n_begin, n_end, s); \
    } else {                                                                             \
      if (sketch_dtype == SAKI_BF16)                                                     \
        launch_build<RK, false, true>(keys, B_k, mu, B, H_q, H_kv, N_cap, ix, n_begin, n_end, s); \
      else                                                                               \
        launch_build<RK, false, false>(keys, B_k, mu, B, H_q, H_kv, N_cap, ix, n_begin, n_end, s); \
    }                                                                                    \
  } while (0)
  switch (r) {
    case 16: SAKI_BUILD(16); break;
    case 32: SAKI_BUILD(32); break;
    case 64: SAKI_BUILD(64); break;
    default: SAKI_BUILD(128); break;
  }
#undef SAKI_BUILD
  return launch_ok() ? SAKI_OK : SAKI_ERR_HIP;
}

int saki_index_export(const void* index, int sketch_dtype, int B, int H_q, int N_cap, int r,
                      float* out, void* stream) {
  if (!index || !out || B <= 0 || H_q <= 0 || N_cap < 0) return SAKI_ERR_ARG;
  if ((long long)B * H_q > 65535) return SAKI_ERR_UNSUPPORTED;
  if (!dtype_ok(sketch_dtype) || !saki::rank_supported(r)) return SAKI_ERR_UNSUPPORTED;
  if (N_cap == 0) return SAKI_OK;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  dim3 grid((unsigned)saki::n_tiles(N_cap), B * H_q);
  const uint8_t* ix = reinterpret_cast<const uint8_t*>(index);
  const int nt = (int)saki::n_tiles(N_cap);
#define SAKI_EXPORT(RK)                                                                       \
  do {                                                                                        \
    if (sketch_dtype == SAKI_BF16)                                                            \
      hipLaunchKernelGGL((export_kernel<RK, true>), grid, dim3(64), 0, s, ix, nt, N_cap, out);  \
    else                                                                                      \
      hipLaunchKernelGGL((export_kernel<RK, false>), grid, dim3(64), 0, s, ix, nt, N_cap, out); \
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

int saki_score_topk(const void* index, int sketch_dtype, int B, int H_q, int H_kv, int N_cap,
                    int N_valid, int d, int r, const float* q, const int* q_pos, int Q,
                    const float* B_q, const float* mu, int k, int* top_idx, float* top_score,
                    void* ws, size_t ws_bytes, void* stream) {
  int st = check_common(B, H_q, H_kv, N_cap, N_valid, d);
  if (st != SAKI_OK) return st;
  if (Q < 0) return SAKI_ERR_ARG;
  if (!dtype_ok(sketch_dtype) || !saki::rank_supported(r) || k < 1 || k > kMaxK)
    return SAKI_ERR_UNSUPPORTED;
  if (Q == 0) return SAKI_OK;
  if (!index || !q || !B_q || !mu || !top_idx || !ws) return SAKI_ERR_ARG;
  const saki::Plan p = saki::score_plan(B, H_q, Q, N_valid, r);
  if (ws_bytes < p.ws_bytes) return SAKI_ERR_WORKSPACE;
  if ((size_t)p.row_blocks * p.n_chunks > 0x7fffffffu) return SAKI_ERR_UNSUPPORTED;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const uint8_t* ix = reinterpret_cast<const uint8_t*>(index);
  uint8_t* w = reinterpret_cast<uint8_t*>(ws);
#define SAKI_SCORE(RK)                                                                        \
  do {                                                                                        \
    if (sketch_dtype == SAKI_BF16)                                                            \
      launch_score<RK, true>(ix, B, H_q, H_kv, N_cap, N_valid, q, q_pos, Q, B_q, mu, k,       \
                             top_idx, top_score, w, p, s);                                    \
    else                                                                                      \
      launch_score<RK, false>(ix, B, H_q, H_kv, N_cap, N_valid, q, q_pos, Q, B_q, mu, k,      \
                              top_idx, top_score, w, p, s);                                   \
  } while (0)
  switch (r) {
    case 16: SAKI_SCORE(16); break;
    case 32: SAKI_SCORE(32); break;
    case 64: SAKI_SCORE(64); break;
    default: SAKI_SCORE(128); break;
  }
#undef SAKI_SCORE
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
  const saki::Plan p = saki::recall_plan(B, H_q, Q, N_valid);
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

}  // extern "C"
