// Internal layout and launch planning shared by the host helpers and the HIP
// launchers of libsaki.  Not part of the public ABI.
#pragma once

#include <cstddef>
#include <cstdint>

namespace saki {

constexpr int kHeadDim = 128;  // d on the GPU path
constexpr int kMaxK = 64;      // top-k lists hold 64 entries, one per wave lane
constexpr int kTile = 64;      // keys per index tile
constexpr int kChunkBytes = 16;
constexpr int kScanWaves = 1;          // waves per work-group of the one-pass MFMA scoring kernel
constexpr int kScanMinKeys = 16384;    // rows at least this long take it
constexpr int kBatchMaxChunk = 4096;   // keys per chunk of the two-pass MFMA scoring kernel
constexpr int kBatchWaves = 1;         // its waves per work-group (16 rows each)

inline bool rank_supported(int r) { return r == 16 || r == 32 || r == 64 || r == 128; }
// bytes per code element: float32 (0), bf16 (1), fp8 E4M3 (2)
inline int elem_bytes(int dtype) { return dtype == 2 ? 1 : dtype == 1 ? 2 : 4; }
inline size_t n_tiles(int N) { return ((size_t)N + kTile - 1) / kTile; }
inline size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Index layout, per (sequence b, query head h): tiles of 64 keys; inside a
// tile, the code of key t is cut into 16-byte pieces and piece p of all 64
// keys is stored contiguously:
//   byte offset = ((b*H_q + h)*n_tiles + tile)*64*r*es + p*64*16 + t*16 + e*es
// so a wave that reads piece p of 64 consecutive keys reads 1 KiB contiguously.
inline size_t tile_bytes(int r, int dtype) { return (size_t)kTile * r * elem_bytes(dtype); }
inline size_t index_bytes(int B, int H_q, int N_cap, int r, int dtype) {
  return (size_t)B * H_q * n_tiles(N_cap) * tile_bytes(r, dtype);
}

// How saki_score_topk / saki_recall split the work.  Each wave owns `rows`
// consecutive query rows of one (b, h) and one key chunk; when a row's keys
// are split over several chunks each chunk writes a partial top-64 to the
// workspace and a merge pass reduces them.
struct Plan {
  bool mfma = false;   // 16-row MFMA kernels (Q >= 16) or the streaming kernels
  int rows = 1;        // query rows per wave
  int waves = 1;       // waves per workgroup
  int row_blocks = 0;  // workgroups along the query axis
  bool split = false;  // streaming: the waves of a workgroup share rows and take consecutive chunks
  bool scan = false;   // MFMA rows scored in one pass (row_blocks: 16-row blocks, one per wave;
                       // with a split key axis z_off: chunk gates, flag_off: rows to redo)
  int chunk = kTile;   // keys per chunk (multiple of 64)
  int n_chunks = 1;
  size_t z_off = 0, b_off = 0, part_off = 0, flag_off = 0, ws_bytes = 0;
  size_t flag_count = 0;  // flags per tier (recall path)
};

// `heads` groups of `Q` rows each (the rows of one group read the same codes).
inline Plan make_plan(int B, int heads, int Q, int N_valid, int part_entry_bytes, bool mfma) {
  Plan p;
  p.mfma = mfma;
  p.rows = p.mfma ? 16 : (Q >= 4 ? 4 : 1);
  const int wave_rows = (Q + p.rows - 1) / p.rows;
  const int H_q = heads;
  const int max_waves = p.mfma ? 2 : 4;  // workgroup size of the kernels
  p.waves = wave_rows < max_waves ? (wave_rows < 1 ? 1 : wave_rows) : max_waves;
  p.row_blocks = (Q + p.rows * p.waves - 1) / (p.rows * p.waves);
  const size_t total_waves = (size_t)B * H_q * wave_rows;
  const size_t n = N_valid > 0 ? (size_t)N_valid : 1;
  size_t chunk = round_up(n, kTile);
  // waves wanted over the whole GPU before the key axis is split too
  const size_t target = p.mfma ? 2048 : 8192;
  if (total_waves > 0 && total_waves < target) {
    const size_t want = (target + total_waves - 1) / total_waves;
    size_t c = round_up((n + want - 1) / want, kTile);
    if (c < 2048) c = 2048;
    if (c < chunk) chunk = c;
  }
  p.chunk = (int)chunk;
  p.n_chunks = (int)((n + chunk - 1) / chunk);
  const size_t rows_total = (size_t)B * H_q * Q;
  size_t off = 0;
  if (p.n_chunks > 1) {
    p.part_off = off;
    off = round_up(off + rows_total * p.n_chunks * kMaxK * part_entry_bytes, 256);
  }
  p.ws_bytes = off;
  return p;
}

// Score path: the workspace holds the partial lists of a split key axis
// (float score + int index), at least 256 bytes so that a size of 0 keeps
// meaning invalid arguments.  The MFMA kernels take 16 queries of one head per
// wave (the one-pass kernel when the rows are long); the streaming kernel
// takes the rows of one code set: the H_q / index_heads heads sharing it,
// times Q.  The two-pass MFMA kernel reads the query sketches z (r values per
// row: bf16 for bf16 and fp8 codes (dtype 1, 2), float32 for float32 codes)
// at z_off and b = q . mu (one float per row) at b_off, written by a kernel
// before it; the other kernels form the sketch themselves.
inline Plan score_plan(int B, int H_q, int index_heads, int Q, int N_valid, int r, int dtype) {
  const bool mfma = Q >= 16;
  Plan p = mfma ? make_plan(B, H_q, Q, N_valid, 8, true)
                : make_plan(B, index_heads, (H_q / index_heads) * Q, N_valid, 8, false);
  if (mfma && N_valid >= kScanMinKeys) {
    p.scan = true;
    p.waves = kScanWaves;
    p.row_blocks = (Q + 15) / 16;
    if (p.n_chunks > 1) {  // per (row, chunk) gate of a chunk that kept too few keys; per-row redo flags
      const size_t rows_total = (size_t)B * H_q * Q;
      p.z_off = round_up(p.ws_bytes, 256);
      p.flag_off = round_up(p.z_off + rows_total * p.n_chunks * sizeof(float), 256);
      p.flag_count = rows_total;
      p.ws_bytes = round_up(p.flag_off + rows_total * sizeof(int), 256);
    }
  }
  if (mfma && !p.scan) {  // the two-pass kernel: chunks of at most kBatchMaxChunk keys
    p.waves = kBatchWaves;
    p.row_blocks = ((Q + 15) / 16 + kBatchWaves - 1) / kBatchWaves;
    const size_t n = N_valid > 0 ? (size_t)N_valid : 1;
    if ((size_t)p.chunk > (size_t)kBatchMaxChunk) {
      p.chunk = kBatchMaxChunk;
      p.n_chunks = (int)((n + kBatchMaxChunk - 1) / kBatchMaxChunk);
    }
    const size_t rows_total = (size_t)B * H_q * Q;
    p.part_off = 0;
    p.z_off = p.n_chunks > 1 ? round_up(rows_total * p.n_chunks * kMaxK * 8, 256) : 0;
    p.b_off = round_up(p.z_off + rows_total * r * (dtype == 0 ? 4 : 2), 256);
    p.ws_bytes = round_up(p.b_off + rows_total * sizeof(float), 256);
  }
  const int wave_rows = (int)((H_q / index_heads) * (size_t)Q + p.rows - 1) / p.rows;
  if (!mfma && wave_rows < 4) {  // too few rows to fill a workgroup: its waves split the keys
    p.split = true;
    p.waves = 4;
    p.row_blocks = wave_rows < 1 ? 1 : wave_rows;
  }
  if (p.ws_bytes < 256) p.ws_bytes = 256;
  return p;
}

// Recall path: partial lists hold a double score and an int index (16 bytes
// with padding).  The MFMA path also keeps the keys split into bf16 hi and lo
// parts in tile layout (z_off), the key norm bounds in rows of n_tiles * 64
// (b_off) and two arrays of one flag per wave (flag_off) through which each
// tier hands the waves it could not finish to the next.
inline Plan recall_plan(int B, int H_q, int H_kv, int Q, int N_valid) {
  Plan p = make_plan(B, H_q, Q, N_valid, 16, Q >= 16);
  if (!p.mfma) return p;
  const size_t nt = n_tiles(N_valid);
  p.z_off = round_up(p.ws_bytes, 256);
  p.b_off = round_up(p.z_off + 2 * (size_t)B * H_kv * nt * kTile * kHeadDim * 2, 256);
  p.flag_off = round_up(p.b_off + (size_t)B * H_kv * nt * kTile * sizeof(float), 256);
  const size_t blocks = (size_t)p.row_blocks * p.n_chunks * B * H_q;
  p.flag_count = (blocks + 8) * 2;
  p.ws_bytes = round_up(p.flag_off + 2 * p.flag_count * sizeof(int), 256);
  return p;
}

}  // namespace saki
