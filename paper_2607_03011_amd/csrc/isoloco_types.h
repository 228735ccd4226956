// Device-visible tables shared by the host planner and the HIP kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace isoloco {

// Tile shape of the batched matrix-product kernels (output BM x BN, K slab BK).
constexpr int kBM = 128;
constexpr int kBN = 128;
constexpr int kBK = 16;
constexpr int kGemmThreads = 256;

// Elements per workgroup of the streaming kernels (reduction, trace, write-back).
constexpr int kChunk = 4096;
constexpr int kStreamThreads = 256;

constexpr int kMaxWorkers = 128;

// Most K slices of a split Gram product.
constexpr int kMaxKSplit = 6;

// Schedule classes of the polar iteration: tall matrices (m >= 2n), whose
// smallest singular value stays well away from zero for noise-like spectra,
// and the others (square-ish, where it does not).
constexpr int kSchedClasses = 2;
constexpr int kSchedSquare = 0;
constexpr int kSchedTall = 1;

// One corrected matrix.  "Tall" coordinates: X is m x n with m >= n, stored
// column-major: X[r][c] at ws_off + r + c * m in the workspace buffers.  A
// tensor stored wide is then in its own row-major layout, a square one in
// its row-major bytes (read column-major they are its transpose, whose polar
// factor is the transposed one: the same bytes), and a tall one (rows >
// cols) is transposed tile by tile by the streaming kernels.
struct MatInfo {
  int64_t ws_off;    // element offset in the Delta / X buffers (64-element aligned)
  int64_t src_off;   // element offset in theta / momentum / workers
  int64_t sq_off;    // element offset of this matrix's n x n buffers (Gram, polynomial)
  int64_t part_off;  // element offset of the split-K Gram partials (ksplit * n * n)
  int32_t m, n;      // tall shape
  int32_t ksplit;    // number of K slices of the Gram product (1 = no split)
  int32_t kchunk;    // rows of X per K slice (multiple of kBK)
  int32_t vec;       // 1 if m and n are multiples of 4 (vector loads allowed)
  int32_t tensor;    // index in the caller's layout
  int32_t chunk_begin, chunk_end;  // range of this matrix in the chunk table
  int32_t wide;      // 1 if the tensor is stored wide (rows < cols)
  int32_t sched;     // schedule class (kSchedSquare or kSchedTall)
  int32_t norm_off;  // first of this matrix's gram_tiles(n) Gram-norm partials
  int32_t cnt_off;   // split-K Gram: first of its gram_tiles(n) arrival counters (-1 if not split)
};

// Output tiles of a symmetric n x n product that are computed: those on or
// above the diagonal of the 128 x 128 tiling, tile (tm, tn) with tm <= tn at
// index gram_tile_index(n, tm, tn).
__host__ __device__ inline int gram_tiles(int n) {
  const int T = (n + kBM - 1) / kBM;
  return T * (T + 1) / 2;
}
__host__ __device__ inline int gram_tile_index(int n, int tm, int tn) {
  const int T = (n + kBM - 1) / kBM;
  return tm * T - tm * (tm - 1) / 2 + (tn - tm);
}

// Work item of the streaming kernels: a run of at most kChunk elements of one
// tensor, or a tile of at most kTileRows x kTileCols elements.
// rows == 0: a contiguous run, element i at src + i (stored) and ws + i
// (workspace).  rows > 0: a rows x cols tile (rows <= kTileRows, cols <=
// kTileCols) of a tall tensor stored row-major and iterated column-major:
// element (r, c) of the tile at src + r * src_ld + c as stored and at
// ws + c * ws_ld + r in the workspace.
struct Chunk {
  int64_t src;    // first element, index into theta / momentum / workers
  int64_t ws;     // first element in the workspace buffers (-1 for AVG tensors)
  int32_t count;  // elements
  int32_t mat;    // matrix index, or -1 for AVG tensors
  int32_t vec;    // 1 if every stream allows 16-byte vector access (runs: from src and ws;
                  // tiles: rows, cols, src_ld and ws_ld multiples of 4 and aligned starts)
  int32_t rows, cols;     // tile shape (rows == 0: a contiguous run)
  int32_t src_ld, ws_ld;  // tile strides: the tensor's columns, the iterate's rows
  int32_t pad;
};
// 32 x 256 tiles: a row segment is 1 KB of every stream (one wave's load)
// and a column segment of the iterate 128 bytes (109.5M workload's
// reduction: 5.60 TB/s against 5.48 with 32 x 128 and 5.38 with 16 x 256)
constexpr int kTileRows = 32;
constexpr int kTileCols = 256;

// Bits of MatScalars::flags (the values of the ISOLOCO_FLAG_* constants).
constexpr int kFlagNonfinite = 1;        // Delta had a non-finite value
constexpr int kFlagZero = 2;             // Delta == 0
constexpr int kFlagNotConverged = 4;     // Q^T Q - I above 1e-3 after the last step
constexpr int kFlagBelowResolution = 8;  // smallest singular value below the float32 resolution
constexpr int kFlagInput = kFlagNonfinite | kFlagZero;  // properties of the input itself

// Per-matrix scalars kept in the workspace.
struct MatScalars {
  float fro;        // ||Delta||_F
  float inv_fro;    // 1 / ||Delta||_F (0 for a zero or non-finite matrix)
  float gscale;     // ||X0^T X0||_F^(-1/2): maps sigma_max of X0 = Delta / ||Delta||_F to <= 1
  float sigma_bar;  // <Q, Delta>_F / n
  float resid;      // ||Q^T Q - I||_F / sqrt(n), or -1 if not computed
  int32_t flags;    // ISOLOCO_FLAG_* bits
  int32_t steps;    // polar steps this matrix has taken
  int32_t active;   // 1 while the matrix still iterates (cleared when a phase end stops it)
  int32_t qbuf;     // which X buffer holds the final polar factor
};

// Work item of a batched matrix product: one output tile of one matrix.
struct Task {
  int32_t mat;     // matrix index; -1 marks an empty task that returns at once
  int32_t tm, tn;  // tile row / column
  int32_t ks;      // K slice (Gram only)
};

struct WorkerPtrs {
  const void* p[kMaxWorkers];
};

}  // namespace isoloco
