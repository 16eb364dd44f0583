// Internal descriptors shared by the host planner (HIP-free) and the gfx950 kernels.
//
// Device state block (one per context, allocated by the caller), regions in order, each
// 256-byte aligned:
//   E arena   fp32, one slot per gradient-bucket element (vector slots unused); the E of a
//             matrix sits at its bucket's E base + its offset in the gradient bucket.  After
//             a Q-step it holds F = M + E_prev and E = F - P_hat Q_loc^T is implied (deferred).
//   factors   fp32 per compressed matrix: P (n x r), Q (m x r), Ph (n x r), Qh (m x r),
//             Ql (m x r), all row-major.
//   W         fp64 r x r per matrix: the upper-triangular map with orth(X) = X W for the
//             factor that the next step orthogonalises.
//   gpart     fp64 Gram partial sums, r x r per slice of factor rows.
//   qpart     fp32 Q-step partial products, per row chunk: m_pad x r.
//   counters  u32 arrival counters of the last-block reductions.
//   tables    MatDesc[], VecDesc[], Tile[] for every launch.
#pragma once

#include <cstdint>

namespace acp {

constexpr int kBlock = 256;       // threads per workgroup (4 waves of 64)
constexpr int kWave = 64;
constexpr double kTau = 1e-4;     // rank-deficiency threshold of orth()

struct MatDesc {
  int64_t grad_off;   // offset of the matrix in its gradient bucket (floats)
  int64_t e_off;      // offset of its E slot in the E arena (floats)
  int64_t fac_off_p;  // offset in the P-step factor buffer
  int64_t fac_off_q;  // offset in the Q-step factor buffer
  int64_t p_slot, q_slot, ph_slot, qh_slot, ql_slot;  // float offsets in the factor region
  int64_t w_slot;     // double offset in the W region
  int64_t gpart;      // double offset in the Gram-partial region
  int64_t qpart;      // float offset in the Q-partial region
  int32_t n, m;
  int32_t ctr_gram;   // counter index of the Gram reduction
  int32_t ctr_q;      // first counter index of the Q-step reductions (one per column block)
  int32_t q_rows;     // rows per Q-step row chunk
  int32_t q_chunks;   // number of Q-step row chunks
  int32_t q_cb;       // Q-step column-block width
  int32_t fact_rows;  // factor rows per Gram slice
  int32_t wpr;        // waves per row in the fused P-step
  int32_t pad;
};

struct VecDesc {
  int64_t grad_off, fac_off_p, fac_off_q, numel;
};

enum TileKind : int32_t { T_ROWS = 0, T_FACT = 1, T_VEC = 2, T_QTILE = 3 };

// kind T_ROWS: idx = matrix, a = first row, b = row count
// kind T_FACT: idx = matrix, a = slice, b = slice count
// kind T_VEC : idx = vector, a = first element, b = element count
// kind T_QTILE: idx = matrix, a = row chunk, b = column block
struct Tile {
  int32_t kind, idx, a, b;
};

enum KernelId : int32_t {
  K_APPLY = 0,   // Xh = X W (orthogonalise the reused factor)
  K_PFUSED,      // P-step, one pass: P = M' Qh, E = M' - P Qh^T, raw vectors packed
  K_PROW,        // P-step, general: P = M' Qh, one workgroup per row
  K_EUPD,        // P-step, general: E = M' - P Qh^T
  K_QSTEP,       // Q-step: F = M', Q = M'^T Ph (deterministic two-level sum), raw vectors packed
  K_RECON,       // decompress: M_hat = P Q^T / p, factor kept + Gram -> W, raw vectors / p
  K_GRAM,        // Gram -> W of a factor slot (after bind / restore)
  K_EMAT,        // materialise E into a bucket-shaped buffer
  K_VEC,         // pack raw vectors only
};

struct Launch {
  int32_t kernel;
  int32_t variant;   // kernel-specific: column slots per lane (K_PFUSED), vector width (K_QSTEP,
                     // K_RECON, K_EMAT, K_EUPD), factor P=0 / Q=1 (K_APPLY, K_GRAM)
  int64_t tile_off;  // first tile in the tile table
  int32_t ntiles;
  int32_t pad;
};

// Kernel arguments (passed by value).
struct KArgs {
  const float* grad;    // gradient bucket (compress)
  float* fbuf;          // factor buffer (compress writes)
  const float* agg;     // aggregated factor buffer (decompress reads)
  float* out;           // output bucket (decompress / E export)
  float* e;             // E arena
  float* fac;           // factor region
  double* w;            // W region
  double* gpart;        // Gram partials
  float* qpart;         // Q-step partials
  uint32_t* ctr;        // counters
  const MatDesc* mats;
  const VecDesc* vecs;
  const Tile* tiles;    // this launch's tiles
  int32_t ntiles;
  int32_t variant;
  int32_t ef;           // error feedback on
  int32_t deferred;     // E arena holds F (E implied) for this bucket
  float inv_p;          // 1 / world size
  int32_t parity;       // 1 on odd (P-) steps, 0 on even (Q-) steps
};

}  // namespace acp
