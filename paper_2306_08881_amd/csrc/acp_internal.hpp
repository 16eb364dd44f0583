// Internal descriptors shared by the host planner (HIP-free) and the gfx950 kernels.
//
// Device state block (one per context, allocated by the caller), regions in order, each
// 256-byte aligned:
//   E arena   fp32, one slot per gradient-bucket element (vector slots unused); the E of a
//             matrix sits at its bucket's E base + its offset in the gradient bucket.  After
//             a Q-step it holds F = M' and E = F - P_hat Q_loc^T is implied (deferred).  After
//             a P-step of rank >= 8 it holds X = M' and E = X - P_loc Q_hat^T is implied
//             (P-deferred); after a P-step of rank <= 4 it holds E itself.
//   factors   fp32 per compressed matrix: P (n x r), Ph (n x r), Pl (n x r), Q (m x r),
//             Qh (m x r), Ql (m x r), all row-major.  P / Q hold the aggregated factor of
//             the last step that produced it, Ph / Qh the orthogonalised factors, Pl / Ql the
//             local factor of the last P- / Q-step.
//   W         fp64 r x r per matrix: the upper-triangular map with orth(X) = X W for the
//             factor that the next step orthogonalises.
//   gpart     fp64 Gram partial sums, r x r per slice of factor rows (factors of more than one
//             slice only).
//   qpart     fp32 Q-step partial products, per row chunk: m_pad x r.
//   tables    MatDesc[], VecDesc[], Tile[] for every launch.
// No kernel communicates across workgroups: every reduction that spans workgroups is
// finished by a later kernel in the same stream.
#pragma once

#include <cstdint>

namespace acp {

constexpr int kBlock = 256;       // threads per workgroup (4 waves of 64)
constexpr int kWave = 64;
constexpr double kTau = 1e-4;     // rank-deficiency threshold of orth()
constexpr int kMaxTileRows = 256; // rows per tile of the rank-4 row kernels (factor rows in LDS)
// K_QFIN entries (e = column * r + rank, over the whole matrix) per tile: one thread per entry
// for up to 8 row chunks, 4 threads for up to 32, 8 for up to 64 (so that no thread adds more
// than 8 chunks, all requested at once), 16 threads beyond
constexpr int qfin_entries(int32_t q_chunks) {
  return q_chunks <= 8 ? 1024 : (q_chunks <= 32 ? 64 : (q_chunks <= 64 ? 32 : 16));
}
constexpr int64_t kMaxCols = int64_t(1) << 24;  // columns of a compressed matrix, at most
constexpr int kSmallRows = 256;  // T_SMALL matrices: rows (their P rows sit in LDS)
constexpr int kSmallCols = 512;  // T_SMALL matrices: columns (their Q rows sit in LDS)
constexpr int kReconRows = 4;   // rows per tile of the rank-4 decompress
constexpr int kQRows = 256;       // rows per Q-step row chunk (at most; the chunk's Ph rows sit in LDS)
// Size of the static device array that holds one bucket's Q-step partials for the compress entry
// point that allocates nothing (acp_compress_noalloc); a bucket that needs more is refused.
constexpr int64_t kScratchBytes = int64_t(32) << 20;

struct MatDesc {
  int64_t grad_off;   // offset of the matrix in its gradient bucket (floats)
  int64_t e_off;      // offset of its E slot in the E arena (floats)
  int64_t fac_off_p;  // offset in the P-step factor buffer
  int64_t fac_off_q;  // offset in the Q-step factor buffer
  int64_t p_slot, q_slot, ph_slot, qh_slot, ql_slot, pl_slot;  // float offsets in the factor region
  int64_t w_slot;     // double offset in the W region
  int64_t gpart;      // double offset in the Gram-partial region
  int64_t qpart;      // float offset in the Q-partial region
  int32_t n, m;
  int32_t q_rows;     // rows per Q-step row chunk
  int32_t q_chunks;   // number of Q-step row chunks
  int32_t q_cb;       // Q-step column-block width
  int32_t fact_rows;  // factor rows per Gram slice
  int32_t scls;       // column class S of the rank-4 kernels (64 S float4 groups per wave)
  int32_t bucket;     // bucket index
  int32_t fact_slices_p, fact_slices_q;  // Gram slices of the P / Q factor rows
  int32_t q_grp;      // Q-step row chunks whose rows interleave (see q_chunk_rows)
  int32_t tid;        // registration index of the tensor (keys the no-reuse draws)
};

// the planner (host compiler) and the kernels (hipcc) share the chunk geometry below
#ifdef __HIPCC__
#define ACP_HOST_DEVICE __host__ __device__
#else
#define ACP_HOST_DEVICE
#endif

// Rows of Q-step row chunk c: chunks go in groups of q_grp that share q_grp * q_rows rows (the
// last group: its rows over q_rows, rounded up), chunk x of a group of g taking rows
// x, x + g, x + 2g, ... of it.  q_grp = 1: chunk c is rows [c q_rows, (c + 1) q_rows).
struct ChunkRows {
  int64_t first;
  int32_t stride, rows;
};
ACP_HOST_DEVICE inline ChunkRows q_chunk_rows(const MatDesc& d, int64_t c) {
  const int64_t gi = c / d.q_grp;
  const int64_t span = int64_t(d.q_grp) * d.q_rows;
  const int64_t base = gi * span;
  const int64_t rem = (d.n - base) < span ? (d.n - base) : span;
  const int64_t g = (rem + d.q_rows - 1) / d.q_rows;
  const int64_t x = c - gi * d.q_grp;
  return ChunkRows{base + x, static_cast<int32_t>(g), static_cast<int32_t>((rem - x + g - 1) / g)};
}

struct VecDesc {
  int64_t grad_off, fac_off_p, fac_off_q, numel;
  int64_t e_off;      // its slot in the E arena (Power-SGD's image of M' holds the raw vector there)
  int32_t bucket, pad;
};

enum TileKind : int32_t { T_ROWS = 0, T_FACT = 1, T_VEC = 2, T_QTILE = 3, T_SROWS = 4, T_SMALL = 5 };

// kind T_ROWS : idx = matrix, a = first row, b = row count (K_APPLY from kApplyMfmaRank on: + 65536 x
//               the 64-column block of Xh)
// kind T_SMALL: idx = matrix, the whole matrix in one workgroup (rank 4, small matrices whose
//               rows are not 16-byte aligned: n <= kSmallRows, m <= kSmallCols)
// kind T_SROWS: idx = matrix, a = first row, b = cb | stride << 4 | count << 16: columns
//               [1024 cb, 1024 cb + 1024) of rows a + k stride, k < count
// kind T_FACT : idx = matrix, a = slice (+ 65536 x part of the Gram blocks from kBlockedRank
//               on: gram_parts(r) parts), b = slice count; K_GSUM: a = entry block of
//               kGsumEntries, b = slice count
// kind T_VEC  : idx = vector, a = first element, b = element count
// kind T_QTILE: idx = matrix, a = row chunk (K_QSTEP) or entry block (K_QFIN), b = column block;
//               K_IMAGE: a = first row, b = column block | row count << 16 (kImageCols columns)
// K_DRAW      : T_ROWS, idx = matrix, a = first factor row, b = row count
// K_IMAGE     : T_FACT, idx = matrix (W = I); T_VEC as for the vector copies
struct Tile {
  int32_t kind, idx, a, b;
};

enum KernelId : int32_t {
  K_APPLY = 0,   // Xh = X W (orthogonalise the reused factor), general path
  K_PFUSED,      // P-step, one pass (r = 4): Qh = Q W, P = M' Qh, E = M' - P Qh^T, vectors packed
  K_PROW,        // P-step, general: P = M' Qh, one workgroup per row
  K_EUPD,        // P-step, general: E = M' - P Qh^T
  K_QSTEP,       // Q-step: F = M' written back, per-chunk partials of M'^T Ph, vectors packed
  K_QFIN,        // Q-step: Q_loc = sum of the chunk partials -> factor buffer and Ql
  K_RECON,       // decompress, general: M_hat = P Q^T / p; factor tiles; vectors / p
  K_RECON4,      // decompress, r = 4 register-resident columns; factor tiles; vectors / p
  K_FACT,        // factor tiles alone: Gram -> W (after bind / restore)
  K_CHOL,        // sum of a factor's Gram partials (more than one slice) -> W
  K_EMAT,        // materialise E into a bucket-shaped buffer
  K_VEC,         // pack raw vectors only
  K_WPSTEP,      // P-step, ranks 8..32 (MFMA): X = M' written, P_loc = X Qh per 32-row tile
  K_WQSTEP,      // Q-step, ranks 8..32 (MFMA): F = M' written, per-chunk partials of F^T Ph
  K_WRECON,      // decompress, ranks 8..32 (MFMA): M_hat = A B^T / p
  K_WFACT,       // decompress, ranks 8..32: factor tiles and vectors / p
  // tile-size classes of the rank-4 narrow-row tiles (rows of at most 512 columns: several rows
  // per wave); they run inside the K_PFUSED (S = 1), fused K_QSTEP and K_RECON4 launches
  K_PNARROW,
  K_QNARROW,
  K_RNARROW,
  K_GSUM,        // from kBlockedRank on: a factor's Gram partials summed (and mirrored) into the first
  K_DRAW,        // no reuse: a fresh standard normal factor into the P (variant 0) or Q (1) slot
  K_IMAGE,       // Power-SGD: M' = M + E into the E arena (raw vectors too), W = I
};

// Narrow rows (r = 4, m / 4 = m4 <= 128 float4 groups): L lanes per row (16, 32 or 64), G float4
// groups per lane (1 or 2); the launch variant is (L << 4) | G.
constexpr int32_t narrow_variant(int32_t m4) {
  return m4 <= 16 ? (16 << 4) | 1 : m4 <= 32 ? (32 << 4) | 1 : m4 <= 64 ? (64 << 4) | 1 : (64 << 4) | 2;
}

constexpr int32_t kWideRank = 8;   // ranks at or above this take the K_W* kernels
constexpr int32_t kBlockedRank = 128;  // ranks whose W K_CHOL forms from Gram partials in global memory
// ranks whose MFMA compress kernels split the rank over the four waves of a workgroup
// (kSplitRank), whose decompress kernel does (kSplitReconRank), and whose W is factored in
// 2 x 2 blocks of 128 (kCholBlockRank)
constexpr int32_t kSplitRank = 64;
constexpr int32_t kSplitReconRank = 256;
constexpr int32_t kCholBlockRank = 256;
// ranks whose orthogonal factor X W is formed on the fp64 matrix cores (one block of
// min(r, 64) columns per tile; below kBlockedRank a factor has one such block)
constexpr int32_t kApplyMfmaRank = 32;
constexpr int32_t apply_blocks(int32_t r) { return r >= 64 ? r / 64 : 1; }  // column blocks of X W
// tiles that share one slice's Gram from kBlockedRank on: the (r / 64)(r / 64 + 1) / 2 blocks of
// 64 x 64 on and above the diagonal, one per wave of a four-wave tile
constexpr int32_t gram_parts(int32_t r) {
  return r >= kBlockedRank ? ((r / 64) * (r / 64 + 1) / 2 + 3) / 4 : 1;
}
constexpr int32_t kGsumEntries = 4096;  // Gram entries per K_GSUM tile
constexpr int kWideBlock = 64;     // threads per workgroup of K_WPSTEP, K_WQSTEP, K_WRECON: one wave
constexpr int kWideQCols = 32;     // K_WQSTEP column block (one MFMA block)
constexpr int kWidePWaves = 4;     // ranks 8..32: waves of a K_WPSTEP workgroup (adjacent column blocks)
constexpr int kWideQWaves = 4;     // ranks 8..32: waves of a K_WQSTEP workgroup (adjacent column blocks)
constexpr int kWideQRows = 512;    // K_WQSTEP rows per chunk (at most)
constexpr int kWideRCols = 1024;   // K_WRECON columns per tile: 32 blocks of 32
constexpr int kImageCols = 256;    // K_IMAGE columns per tile: one per thread
constexpr int kDrawRows = 256;     // K_DRAW factor rows per tile
// K_IMAGE rows per tile: their row-factor rows sit in LDS (at most 16 KB)
constexpr int image_rows(int32_t r) { return r <= 64 ? 64 : 4096 / r; }

// K_QSTEP variants: column slots per lane | kQFused when the kernel also orthogonalises P
constexpr int32_t kQFused = 16;
// K_PFUSED variant bits: S = 1 on three waves, for rows of 516 to 768 columns; S = 2 on eight
// waves, for rows of 3076 to 4096 columns
constexpr int32_t kThreeWaves = 32;
constexpr int32_t kEightWaves = 64;
// K_FACT variants: bit 0 = Q (else P); bit 1 (kFactFromBuffer): the factor is read from the
// aggregated factor buffer (src) and copied into its slot, else read from its slot
constexpr int32_t kFactFromBuffer = 2;

struct Launch {
  int32_t kernel;
  int32_t variant;   // kernel-specific: column class S (K_PFUSED, K_RECON4), vector width
                     // (K_QSTEP, K_RECON), factor P=0 / Q=1 (K_APPLY, K_FACT)
  int64_t tile_off;  // first tile in the tile table
  int32_t ntiles;
  int32_t family;    // ACP_KERNEL_* family (host-side profiling)
  double alg_bytes;  // algorithmic bytes of the launch (host-side profiling)
};


// Buckets per launch: a launch covers the buckets [base, base + kMaxGroup) at most; their
// buffer addresses travel in the kernel arguments.
constexpr int kMaxGroup = 64;

// Kernel arguments (passed by value).
struct KArgs {
  const float* src[kMaxGroup];  // per bucket: gradient bucket (compress) or aggregated factor
                                // buffer (decompress)
  float* dst[kMaxGroup];        // per bucket: factor buffer (compress), output bucket
                                // (decompress, E export)
  float* e;             // E arena
  float* fac;           // factor region
  double* w;            // W region
  double* gpart;        // Gram partials
  float* qpart;         // Q-step partials
  const MatDesc* mats;
  const VecDesc* vecs;
  const Tile* tiles;    // this launch's tiles
  uint64_t deferred;    // bit i: the E arena of bucket base + i holds F (E implied)
  uint64_t deferred_p;  // bit i: the E arena of bucket base + i holds X (E implied)
  int32_t base;         // bucket of src[0] / dst[0]
  int32_t ntiles;
  int32_t variant;
  int32_t ef;           // error feedback on
  float inv_p;          // 1 / world size
  int32_t parity;       // 1 on odd (P-) steps, 0 on even (Q-) steps
  int32_t copy_only;    // factor tiles copy the aggregated factor but build no W (Power-SGD)
  uint64_t seed;        // K_DRAW: the context's seed
  int64_t step;         // K_DRAW: the step whose factors are drawn
};

}  // namespace acp
