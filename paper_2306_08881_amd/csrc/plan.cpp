// Host planner: reshape and eligibility, tensor-fusion buckets, factor-buffer offsets, state
// regions and the launch tables of every bucket and phase.
//
// Layout rules (arXiv 2306.08881):
//  * Section IV-C: vector-shaped gradients are not compressed, other gradients are reshaped
//    into matrices; the matrix is n = dim 0 by m = product of the other dims.  A matrix with
//    r >= min(n, m) gains nothing from a rank-r factorisation and is passed through too.
//  * Section IV-B, "Buffer Size": buckets of a fixed byte size (25 MB in PyTorch-DDP, read as
//    MiB), filled with whole tensors in backward order (reverse registration order); a bucket
//    is closed once it reaches the cap.
//  * Section IV-B / IV-C: each bucket's factor buffer holds the compressed factors (P: n x r on
//    P-steps, Q: m x r on Q-steps) and the raw vectors, packed in bucket order.
#include "plan.hpp"

#include <algorithm>
#include <array>
#include <climits>
#include <cmath>
#include <map>

namespace acp {

namespace {

constexpr int64_t kTileElems = 16384;   // gradient elements per streaming tile (unit)
constexpr int64_t kSmallTileElems = 2048;  // per tile of the general P-step E update and decompress
constexpr int64_t kTargetTiles = 1024;     // workgroups a launch class aims for (4 per CU)
constexpr int64_t kMinTileElems = 2048;    // smallest tile of a class that has few elements
constexpr int64_t kPGroup = 8;            // P-step tiles whose rows interleave (rank 4)
constexpr int64_t kMergeElems = int64_t(16) << 20;  // P-step classes below this share a launch
constexpr int64_t kPMinRows = 8;          // fewest rows of a P-step tile (rank 4)
constexpr int64_t kQGroup = 8;            // Q-step row chunks whose rows interleave (rank 4)
constexpr int64_t kVecChunk = 4096;     // raw-vector elements per copy tile
constexpr int64_t kApplyRows = 256;     // factor rows per orthogonalisation tile
constexpr int64_t kSlotAlign = 64;      // floats (256 bytes)

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
int64_t align_up(int64_t x, int64_t a) { return cdiv(x, a) * a; }

bool rank_supported(int32_t r) {
  return r == 1 || r == 2 || r == 4 || r == 8 || r == 16 || r == 32 || r == 64 || r == 128 || r == 256;
}

struct TileSink {
  std::vector<Tile>& tiles;
  Launch begin(int32_t kernel, int32_t variant) {
    Launch l{};
    l.kernel = kernel;
    l.variant = variant;
    l.tile_off = static_cast<int64_t>(tiles.size());
    return l;
  }
  void end(Launch& l, std::vector<Launch>& list) {
    l.ntiles = static_cast<int32_t>(static_cast<int64_t>(tiles.size()) - l.tile_off);
    if (l.ntiles > 0) list.push_back(l);
  }
};

}  // namespace

std::string build_plan(Plan& plan, int32_t num_tensors, const int32_t* ndims, const int64_t* dims,
                       int32_t rank, int64_t cap_bytes, bool ef, bool reuse, bool psgd) {
  if (num_tensors <= 0) return "num_tensors must be positive";
  if (!ndims || !dims) return "ndims and dims must not be NULL";
  if (!rank_supported(rank)) return "rank must be one of 1, 2, 4, 8, 16, 32, 64, 128, 256";
  if (cap_bytes <= 0) return "bucket_cap_bytes must be positive";
  if (psgd && !reuse) return "Power-SGD reuses Q";
  plan = Plan{};
  plan.rank = rank;
  plan.cap_bytes = cap_bytes;
  plan.ef = ef;
  plan.reuse = reuse;
  plan.psgd = psgd;
  // Power-SGD runs ACP-SGD's product kernels without error feedback on the image M' = M + E that
  // its first half writes into the E arena: their lists carry no E update of their own
  const bool list_ef = ef && !psgd;
  const int64_t r = rank;

  // ---- tensors: reshape and eligibility
  int64_t di = 0;
  plan.tensors.resize(num_tensors);
  for (int32_t i = 0; i < num_tensors; ++i) {
    const int32_t nd = ndims[i];
    if (nd < 1 || nd > 8) return "tensor " + std::to_string(i) + ": ndims must be in 1..8";
    TensorPlan& t = plan.tensors[i];
    int64_t numel = 1;
    for (int32_t k = 0; k < nd; ++k) {
      const int64_t d = dims[di + k];
      if (d <= 0 || d > (int64_t(1) << 31)) return "tensor " + std::to_string(i) + ": bad dim";
      numel *= d;
      if (numel > (int64_t(1) << 40)) return "tensor " + std::to_string(i) + ": too large";
      t.shape.push_back(d);
    }
    di += nd;
    t.numel = numel;
    if (nd >= 2) {
      const int64_t n = t.shape[0], m = numel / n;
      if (r < std::min(n, m)) {
        // the kernels address a factor of m rows of r floats with 32-bit byte offsets
        if (m > std::min<int64_t>(kMaxCols, ((int64_t(1) << 32) - 1) / (4 * r)))
          return "tensor " + std::to_string(i) +
                 ": compressed matrices may have at most min(2^24, (2^32 - 1) / (4 r)) columns";
        t.compressed = true;
        t.n = n;
        t.m = m;
      }
    }
    if (!t.compressed) {
      // a raw tensor's element offsets travel as 32-bit tile fields
      if (numel > INT32_MAX) return "tensor " + std::to_string(i) + ": raw tensors may have at most 2^31 - 1 elements";
      t.n = numel;
      t.m = 1;
    } else if (t.n > INT32_MAX) {
      return "tensor " + std::to_string(i) + ": compressed matrices may have at most 2^31 - 1 rows";
    }
  }

  // ---- buckets: backward order, close once the byte size reaches the cap
  {
    BucketPlan cur;
    int64_t cur_bytes = 0;
    for (int32_t i = num_tensors - 1; i >= 0; --i) {
      TensorPlan& t = plan.tensors[i];
      cur.tids.push_back(i);
      cur.grad_off.push_back(cur.grad_elems);
      cur.fac_off_p.push_back(cur.fac_elems_p);
      cur.fac_off_q.push_back(cur.fac_elems_q);
      cur.grad_elems += t.numel;
      cur.fac_elems_p += t.compressed ? t.n * r : t.numel;
      cur.fac_elems_q += t.compressed ? t.m * r : t.numel;
      cur_bytes += t.numel * 4;
      if (cur_bytes >= cap_bytes) {
        plan.buckets.push_back(std::move(cur));
        cur = BucketPlan{};
        cur_bytes = 0;
      }
    }
    if (!cur.tids.empty()) plan.buckets.push_back(std::move(cur));
  }

  // ---- launch classes of the rank-4 kernels and their total elements: a class with few
  // elements gets smaller tiles, so that its (grouped) launch still has about kTargetTiles
  // workgroups instead of a few long serial ones
  const bool wide = r >= kWideRank;
  std::map<int64_t, int64_t> class_elems;
  auto class_key = [](int32_t kernel, int32_t variant) { return int64_t(kernel) * 65536 + variant; };
  // (P-step kernel, variant), (Q-step kernel, variant), (decompress kernel, variant) of a
  // rank-4 matrix that the register-resident kernels take; kernel -1 for the general path
  auto rank4_classes = [&](int64_t m, int64_t grad_off, int64_t fac_p, int64_t fac_q) {
    std::array<std::pair<int32_t, int32_t>, 3> c{};
    const bool fast = r == 4 && m % 4 == 0 && grad_off % 4 == 0 && fac_p % 4 == 0 && fac_q % 4 == 0 &&
                      cdiv(m / 4, 256) <= 5;
    if (!fast) {
      c.fill({-1, 0});
    } else if (m / 4 <= 128) {
      const int32_t v = narrow_variant(static_cast<int32_t>(m / 4));
      c = {{{K_PNARROW, v}, {K_QNARROW, v}, {K_RNARROW, v}}};
    } else if (m / 4 <= 192) {  // three waves cover a row of the P-step
      c = {{{K_PFUSED, 1 | kThreeWaves}, {K_QSTEP, 4 | kQFused}, {K_RECON4, 0}}};
    } else if (m / 4 > 768 && m / 4 <= 1024) {  // eight waves of two groups cover a row
      c = {{{K_PFUSED, 2 | kEightWaves}, {K_QSTEP, 4 | kQFused}, {K_RECON4, 0}}};
    } else {
      const int32_t S = static_cast<int32_t>(cdiv(m / 4, 256));
      c = {{{K_PFUSED, S}, {K_QSTEP, 4 | kQFused}, {K_RECON4, 0}}};
    }
    return c;
  };
  for (const BucketPlan& bk : plan.buckets)
    for (size_t k = 0; k < bk.tids.size(); ++k) {
      const TensorPlan& t = plan.tensors[bk.tids[k]];
      if (!t.compressed || wide) continue;
      for (const auto& kv : rank4_classes(t.m, bk.grad_off[k], bk.fac_off_p[k], bk.fac_off_q[k]))
        if (kv.first >= 0) class_elems[class_key(kv.first, kv.second)] += t.n * t.m;
    }
  // elements per tile of a class: its total over kTargetTiles, between kMinTileElems and `base`
  auto class_tile = [&](int32_t kernel, int32_t variant, int64_t base) {
    const auto it = class_elems.find(class_key(kernel, variant));
    const int64_t tot = it == class_elems.end() ? 0 : it->second;
    return std::max<int64_t>(kMinTileElems, std::min<int64_t>(base, tot / kTargetTiles));
  };

  // P-step launch classes: a class S >= 2 with fewer than kMergeElems elements in all runs in
  // one launch with the other such classes, as the largest of them (pmerge; 0: none)
  int32_t pmerge = 0;
  for (int32_t S = 2; S <= 5; ++S) {
    const auto it = class_elems.find(class_key(K_PFUSED, S));
    if (it != class_elems.end() && it->second > 0 && it->second < kMergeElems) pmerge = S;
  }
  auto class_of_p = [&](int32_t S) -> int32_t {
    if (S < 2 || pmerge == 0) return S;
    const auto it = class_elems.find(class_key(K_PFUSED, S));
    const int64_t tot = it == class_elems.end() ? 0 : it->second;
    return tot < kMergeElems ? pmerge : S;
  };

  // ---- per-tensor device descriptors and state regions
  int64_t e_floats = 0, fac_floats = 0, gpart = 0, qpart = 0;
  for (int32_t b = 0; b < static_cast<int32_t>(plan.buckets.size()); ++b) {
    BucketPlan& bk = plan.buckets[b];
    bk.e_base = e_floats;
    if (ef) e_floats += align_up(bk.grad_elems, kSlotAlign);
    for (int32_t k = 0; k < static_cast<int32_t>(bk.tids.size()); ++k) {
      TensorPlan& t = plan.tensors[bk.tids[k]];
      t.bucket = b;
      t.pos = k;
      if (!t.compressed) {
        VecDesc v{};
        v.grad_off = bk.grad_off[k];
        v.fac_off_p = bk.fac_off_p[k];
        v.fac_off_q = bk.fac_off_q[k];
        v.numel = t.numel;
        v.e_off = bk.e_base + bk.grad_off[k];
        v.bucket = b;
        t.vec = static_cast<int32_t>(plan.vecs.size());
        bk.vecs.push_back(t.vec);
        plan.vecs.push_back(v);
        continue;
      }
      MatDesc d{};
      d.n = static_cast<int32_t>(t.n);
      d.m = static_cast<int32_t>(t.m);
      d.grad_off = bk.grad_off[k];
      d.e_off = bk.e_base + bk.grad_off[k];
      d.fac_off_p = bk.fac_off_p[k];
      d.fac_off_q = bk.fac_off_q[k];
      d.tid = bk.tids[k];
      const int64_t np = align_up(t.n * r, kSlotAlign), mp = align_up(t.m * r, kSlotAlign);
      d.p_slot = fac_floats;
      d.ph_slot = fac_floats + np;
      d.pl_slot = fac_floats + 2 * np;
      d.q_slot = fac_floats + 3 * np;
      d.qh_slot = d.q_slot + mp;
      d.ql_slot = d.q_slot + 2 * mp;
      fac_floats += 3 * np + 3 * mp;
      const bool vec4 = (t.m % 4 == 0) && (d.grad_off % 4 == 0);
      const int64_t cpt = (vec4 && r <= 8) ? 4 : 1;
      d.q_cb = wide ? kWideQCols : static_cast<int32_t>(4 * 64 * cpt);
      // rows per chunk: kQRows (kWideQRows), fewer when a chunk's byte extent would pass 2^30
      // (the kernels address a tile with 32-bit offsets from the tile's first element)
      d.q_rows = static_cast<int32_t>(std::max<int64_t>(
          1, std::min<int64_t>(wide ? (r >= kBlockedRank ? 4 * kWideQRows : kWideQRows) : kQRows,
                               (int64_t(1) << 30) / (t.m * 4))));
      // a small matrix the general kernels take is split into at least 4 chunks (16 rows or
      // more each), so its Q-step is not one workgroup's serial walk
      const bool fast = r == 4 && vec4 && d.fac_off_p % 4 == 0 && d.fac_off_q % 4 == 0 && t.m / 4 <= 1280;
      if (!wide && !fast)
        d.q_rows = std::min<int32_t>(d.q_rows, std::max<int32_t>(16, static_cast<int32_t>(cdiv(t.n, 4))));
      if (!wide && fast) {
        // chunk rows of a multiple of 16 holding about the class's elements per tile
        const auto qc = rank4_classes(t.m, d.grad_off, d.fac_off_p, d.fac_off_q)[1];
        const int64_t cols = std::min<int64_t>(t.m, d.q_cb);
        const int64_t want = class_tile(qc.first, qc.second, int64_t(kQRows) * cols) / cols;
        d.q_rows = std::min<int32_t>(d.q_rows, static_cast<int32_t>(std::max<int64_t>(16, want / 16 * 16)));
      }
      // the register-resident rank-4 Q-step interleaves the rows of kQGroup chunks (offsets of a
      // chunk stay below 2^31: at most kQGroup * kQRows rows of at most 5120 columns)
      d.q_grp = (!wide && fast && t.m / 4 > 128) ? static_cast<int32_t>(kQGroup) : 1;
      d.q_chunks = static_cast<int32_t>(cdiv(t.n, d.q_rows));
      const int64_t ncb = cdiv(t.m, d.q_cb);
      d.qpart = qpart;
      if (bk.mats.empty()) bk.qpart_base = qpart;
      qpart += align_up(int64_t(d.q_chunks) * ncb * d.q_cb * r, kSlotAlign);
      bk.qpart_floats = qpart - bk.qpart_base;
      d.bucket = b;
      // factor rows per Gram slice: at r <= 8 up to 8192 (one slice, and no K_CHOL, for
      // factors of at most 8192 rows); at r >= 16 at least 256 and at most 32 slices per factor
      // (K_CHOL adds a factor's slice partials in one workgroup); from kBlockedRank on at least
      // 1024, since every slice adds an r x r partial for K_GSUM to read (1024 measured faster
      // than 256, 512, 2048 and 4096), and again at most 32, so that no slice is much longer
      d.fact_rows = r <= 8 ? 8192
                    : r >= kBlockedRank
                        ? static_cast<int32_t>(std::max<int64_t>(1024, align_up(cdiv(std::max(t.n, t.m), 32), 64)))
                        : static_cast<int32_t>(std::max<int64_t>(256, align_up(cdiv(std::max(t.n, t.m), 32), 64)));
      d.fact_slices_p = static_cast<int32_t>(cdiv(t.n, d.fact_rows));
      d.fact_slices_q = static_cast<int32_t>(cdiv(t.m, d.fact_rows));
      d.gpart = gpart;
      {
        const int64_t nsl = std::max(d.fact_slices_p, d.fact_slices_q);
        if (nsl > 1 || r >= kBlockedRank) gpart += nsl * r * r;
      }
      d.w_slot = static_cast<int64_t>(plan.mats.size()) * r * r;
      t.mat = static_cast<int32_t>(plan.mats.size());
      bk.mats.push_back(t.mat);
      plan.mats.push_back(d);
    }
  }

  // ---- launch tables
  TileSink sink{plan.tiles};
  auto vec_tiles = [&](const BucketPlan& bk) {
    for (int32_t v : bk.vecs) {
      const int64_t n = plan.vecs[v].numel;
      for (int64_t s = 0; s < n; s += kVecChunk)
        plan.tiles.push_back(Tile{T_VEC, v, static_cast<int32_t>(s),
                                  static_cast<int32_t>(std::min(kVecChunk, n - s))});
    }
  };
  // orthogonalisation tiles of kApplyRows factor rows; from kApplyMfmaRank on one per column
  // block of Xh as well (b = rows | block << 16)
  auto apply_tiles = [&](const std::vector<int32_t>& mats, bool q) {
    const int32_t ncb = r >= kApplyMfmaRank ? apply_blocks(static_cast<int32_t>(r)) : 1;
    for (int32_t mi : mats) {
      const int64_t rows = q ? plan.mats[mi].m : plan.mats[mi].n;
      for (int64_t s = 0; s < rows; s += kApplyRows)
        for (int32_t cb = 0; cb < ncb; ++cb)
          plan.tiles.push_back(Tile{T_ROWS, mi, static_cast<int32_t>(s),
                                    static_cast<int32_t>(std::min(kApplyRows, rows - s)) | (cb << 16)});
    }
  };
  // factor tiles: one per slice of fact_rows factor rows
  auto fact_tiles = [&](int32_t mi, bool q) {
    const MatDesc& d = plan.mats[mi];
    const int32_t nsl = q ? d.fact_slices_q : d.fact_slices_p;
    const int32_t nq = gram_parts(static_cast<int32_t>(r));
    for (int32_t s = 0; s < nsl; ++s)
      for (int32_t q4 = 0; q4 < nq; ++q4) plan.tiles.push_back(Tile{T_FACT, mi, s + 65536 * q4, nsl});
  };
  // Gram finish of the factors of more than one slice
  auto chol_tiles = [&](int32_t mi, bool q) {
    const MatDesc& d = plan.mats[mi];
    const int32_t nsl = q ? d.fact_slices_q : d.fact_slices_p;
    if (nsl > 1 || r >= kBlockedRank) plan.tiles.push_back(Tile{T_FACT, mi, 0, nsl});
  };
  // from kBlockedRank on: the partials' sum, kGsumEntries Gram entries per tile
  auto gsum_tiles = [&](int32_t mi, bool q) {
    const MatDesc& d = plan.mats[mi];
    const int32_t nsl = q ? d.fact_slices_q : d.fact_slices_p;
    for (int32_t e = 0; e < static_cast<int32_t>(r * r / kGsumEntries); ++e)
      plan.tiles.push_back(Tile{T_FACT, mi, e, nsl});
  };
  // the Gram finish after the factor tiles: K_GSUM from kBlockedRank on, then K_CHOL
  auto chol_launches = [&](const std::vector<int32_t>& mats, bool q, std::vector<Launch>& L) {
    if (r >= kBlockedRank) {
      Launch l = sink.begin(K_GSUM, 0);
      for (int32_t mi : mats) gsum_tiles(mi, q);
      sink.end(l, L);
    }
    Launch l = sink.begin(K_CHOL, 0);
    for (int32_t mi : mats) chol_tiles(mi, q);
    sink.end(l, L);
  };
  auto row_tiles = [&](int32_t mi, int64_t rows_per_tile) {
    const MatDesc& d = plan.mats[mi];
    for (int64_t s = 0; s < d.n; s += rows_per_tile)
      plan.tiles.push_back(Tile{T_ROWS, mi, static_cast<int32_t>(s),
                                static_cast<int32_t>(std::min<int64_t>(rows_per_tile, d.n - s))});
  };
  // rank-4 decompress tiles: 1024-column blocks of kReconRows rows.  Rows go in groups of
  // gr * kReconRows (gr = 8 / column blocks, at least 1); the tiles of a group take rows
  // x, x + gr, x + 2 gr, ... (x < gr) and are ordered (x, block), so that tiles that run together
  // write whole adjacent rows.
  auto recon4_tiles = [&](int32_t mi) {
    const MatDesc& d = plan.mats[mi];
    const int64_t nb = cdiv(d.m, 1024);
    const int64_t gr = std::max<int64_t>(1, 8 / nb);
    for (int64_t g0 = 0; g0 < d.n; g0 += gr * kReconRows) {
      const int64_t end = std::min<int64_t>(d.n, g0 + gr * kReconRows);
      for (int64_t x = 0; x < gr && g0 + x < end; ++x) {
        const int64_t cnt = cdiv(end - g0 - x, gr);
        for (int64_t cb = 0; cb < nb; ++cb)
          plan.tiles.push_back(Tile{T_SROWS, mi, static_cast<int32_t>(g0 + x),
                                    static_cast<int32_t>(cb | (gr << 4) | (cnt << 16))});
      }
    }
  };
  // rank-4 P-step tiles of rows_per_tile rows: groups of kPGroup tiles share kPGroup *
  // rows_per_tile rows, tile x of a group taking rows x, x + g, x + 2g, ... of it (g tiles in the
  // group, kPGroup except in the last one)
  auto pstep_tiles = [&](int32_t mi, int64_t rows_per_tile) {
    const MatDesc& d = plan.mats[mi];
    for (int64_t g0 = 0; g0 < d.n; g0 += kPGroup * rows_per_tile) {
      const int64_t rem = std::min<int64_t>(d.n - g0, kPGroup * rows_per_tile);
      const int64_t g = cdiv(rem, rows_per_tile);
      for (int64_t x = 0; x < g; ++x)
        plan.tiles.push_back(Tile{T_SROWS, mi, static_cast<int32_t>(g0 + x),
                                  static_cast<int32_t>((g << 4) | (cdiv(rem - x, g) << 16))});
    }
  };
  // rank-4 matrices that one workgroup takes whole (T_SMALL) when the row kernels cannot
  auto is_small = [&](int32_t mi) {
    const MatDesc& d = plan.mats[mi];
    return r == 4 && d.n <= kSmallRows && d.m <= kSmallCols;
  };
  auto is_vec4 = [&](int32_t mi) {
    const MatDesc& d = plan.mats[mi];
    return d.m % 4 == 0 && d.grad_off % 4 == 0;
  };
  // rank-4 register-resident kernels: 16-byte aligned rows and factor rows, m <= 5120
  auto is_fast = [&](int32_t mi) {
    const MatDesc& d = plan.mats[mi];
    return r == 4 && is_vec4(mi) && d.fac_off_p % 4 == 0 && d.fac_off_q % 4 == 0 &&
           cdiv(d.m / 4, 256) <= 5;
  };
  // rows per tile of the rank-4 kernels: a multiple of the rows handled per round
  auto rows_for = [&](int32_t mi, int64_t elems) {
    const MatDesc& d = plan.mats[mi];
    const int64_t rb = d.scls == 1 ? 8 : (d.scls <= 4 ? 2 : 1);
    const int64_t rows = rb * std::max<int64_t>(1, elems / (int64_t(d.m) * rb));
    return std::min<int64_t>(rows, kMaxTileRows);
  };

  // Q-step finish tiles: entry blocks of each matrix's column blocks
  auto qfin_launch = [&](const BucketPlan& bk, std::vector<Launch>& L, bool with_vecs) {
    Launch l = sink.begin(K_QFIN, 0);
    for (int32_t mi : bk.mats) {
      const MatDesc& d = plan.mats[mi];
      if (d.scls < 0) continue;  // T_SMALL: the Q-step writes Q_loc itself
      const int64_t nblk = cdiv(int64_t(d.m) * r, qfin_entries(d.q_chunks));
      for (int64_t eb = 0; eb < nblk; ++eb)
        plan.tiles.push_back(Tile{T_QTILE, mi, static_cast<int32_t>(eb), 0});
    }
    if (with_vecs) vec_tiles(bk);
    sink.end(l, L);
  };
  auto emat_launch = [&](BucketPlan& bk) {
    Launch l = sink.begin(K_EMAT, 1);
    for (int32_t mi : bk.mats) row_tiles(mi, std::max<int64_t>(1, kTileElems / plan.mats[mi].m));
    sink.end(l, bk.emat);
  };
  // ranks 8..32: every matrix of the bucket takes the MFMA kernels
  auto wide_lists = [&](BucketPlan& bk) {
    // The compress kernels take matrix tiles, and the raw vectors ride along in the P-step and
    // Q-finish launches; factor tiles go to launches of their own.
    // -- P-step (odd t): Qh = Q W, then 32-row tiles
    {
      std::vector<Launch>& L = bk.compress[1];
      Launch l = sink.begin(K_APPLY, 1);
      apply_tiles(bk.mats, true);
      sink.end(l, L);
      l = sink.begin(K_WPSTEP, 0);
      for (int32_t mi : bk.mats) row_tiles(mi, 32);
      vec_tiles(bk);  // packed by the P-step launch's workgroups
      sink.end(l, L);
    }
    // -- Q-step (even t): Ph = P W, (row chunk, 32-column block) tiles, vectors, finish
    {
      std::vector<Launch>& L = bk.compress[0];
      Launch l = sink.begin(K_APPLY, 0);
      apply_tiles(bk.mats, false);
      sink.end(l, L);
      l = sink.begin(K_WQSTEP, 0);
      for (int32_t mi : bk.mats) {
        const MatDesc& d = plan.mats[mi];
        // below kSplitRank a tile takes kWideQWaves adjacent column blocks, one per wave
        const int32_t per = r < kSplitRank ? kWideQWaves : 1;
        const int32_t ncb = static_cast<int32_t>(cdiv(cdiv(d.m, d.q_cb), per));
        for (int32_t c = 0; c < d.q_chunks; ++c)
          for (int32_t cb = 0; cb < ncb; ++cb) plan.tiles.push_back(Tile{T_QTILE, mi, c, cb});
      }
      sink.end(l, L);
      qfin_launch(bk, L, true);  // the vectors packed by the finish launch's workgroups
    }
    // -- decompress: (32-row block, 512-column group) tiles, then factor tiles and vectors
    for (int32_t par = 0; par < 2; ++par) {
      std::vector<Launch>& L = bk.decompress[par];
      const bool q = par == 0;
      Launch l = sink.begin(K_WRECON, 0);
      for (int32_t mi : bk.mats) {
        const MatDesc& d = plan.mats[mi];
        const int32_t nrb = static_cast<int32_t>(cdiv(d.n, 32));
        const int32_t ncg = static_cast<int32_t>(cdiv(d.m, kWideRCols));
        for (int32_t rb = 0; rb < nrb; ++rb)
          for (int32_t cg = 0; cg < ncg; ++cg) plan.tiles.push_back(Tile{T_QTILE, mi, rb, cg});
      }
      sink.end(l, L);
      l = sink.begin(K_WFACT, 0);
      for (int32_t mi : bk.mats) fact_tiles(mi, q);
      vec_tiles(bk);
      sink.end(l, L);
      chol_launches(bk.mats, q, L);
    }
    emat_launch(bk);
  };

  for (BucketPlan& bk : plan.buckets) {
    if (wide) {
      wide_lists(bk);
      continue;
    }
    // fast: rank-4 register-resident kernels; narrow: rows of at most 512 columns (scls 0);
    // small: rank-4 matrices of other rows, small enough for one workgroup (scls -1, T_SMALL
    // tiles in the same launches); generic: the general kernels
    // three: fast rows of 516-768 columns (three-wave P-step launch)
    // eight: fast rows of 3076-4096 columns (eight-wave P-step launch)
    std::vector<int32_t> fast, narrow, small, generic, three, eight;
    for (int32_t mi : bk.mats) {
      if (is_fast(mi)) {
        const int64_t m4 = plan.mats[mi].m / 4;
        plan.mats[mi].scls = m4 <= 128 ? 0 : static_cast<int32_t>(cdiv(m4, 256));
        (m4 <= 128 ? narrow : (m4 <= 192 ? three : (m4 > 768 && m4 <= 1024 ? eight : fast))).push_back(mi);
      } else if (is_small(mi)) {
        plan.mats[mi].scls = -1;
        small.push_back(mi);
      } else {
        generic.push_back(mi);
      }
    }
    auto small_tiles = [&]() {
      for (int32_t mi : small) plan.tiles.push_back(Tile{T_SMALL, mi, 0, 0});
    };
    auto of_narrow = [&](int32_t v) {
      std::vector<int32_t> out;
      for (int32_t mi : narrow)
        if (narrow_variant(plan.mats[mi].m / 4) == v) out.push_back(mi);
      return out;
    };
    // rows per narrow tile: whole workgroup rounds (256 / L rows), about `elems` elements
    auto narrow_rows = [&](int32_t mi, int64_t elems) {
      const int64_t rw = kBlock / (narrow_variant(plan.mats[mi].m / 4) >> 4);
      return std::min<int64_t>(rw * std::max<int64_t>(1, elems / (int64_t(plan.mats[mi].m) * rw)),
                               kMaxTileRows);  // the decompress stages the tile's A rows in LDS
    };
    const int32_t narrow_vars[4] = {narrow_variant(16), narrow_variant(32), narrow_variant(64),
                                    narrow_variant(128)};
    auto of_class = [&](int32_t S) {
      std::vector<int32_t> v;
      for (int32_t mi : fast)
        if (plan.mats[mi].scls == S) v.push_back(mi);
      return v;
    };
    // -- P-step (odd t)
    {
      std::vector<Launch>& L = bk.compress[1];
      bool vec_done = bk.vecs.empty();
      Launch l = sink.begin(K_APPLY, 1);
      apply_tiles(generic, true);
      sink.end(l, L);
      // the classes S >= 2 with few elements in all (launch variant pmerge) share one launch
      auto pfused_tiles = [&](int32_t S) {
        // rows of 4 KB: 32K elements per tile; rows of 12 KB and more: 64K
        const int64_t base = (S >= 4 ? 4 : 2) * kTileElems;
        for (int32_t mi : of_class(S))
          pstep_tiles(mi, rows_for(mi, std::max<int64_t>(kPMinRows * plan.mats[mi].m,
                                                          class_tile(K_PFUSED, S, base))));
      };
      for (int32_t S = 1; S <= 5; ++S) {
        const bool merged = S >= 2 && class_of_p(S) != S;
        if (merged || (S == pmerge && S >= 2)) continue;  // the merged launch follows
        if (of_class(S).empty() && (S > 1 || (narrow.empty() && small.empty()))) continue;
        l = sink.begin(K_PFUSED, S);
        if (S == 1) {  // the narrow-row and small matrices' tiles ride in the S = 1 launch
          small_tiles();
          for (int32_t v : narrow_vars)
            for (int32_t mi : of_narrow(v)) row_tiles(mi, narrow_rows(mi, class_tile(K_PNARROW, v, 2 * kTileElems)));
        }
        pfused_tiles(S);
        if (!vec_done) vec_tiles(bk), vec_done = true;
        sink.end(l, L);
      }
      if (!three.empty()) {
        l = sink.begin(K_PFUSED, 1 | kThreeWaves);
        for (int32_t mi : three)
          pstep_tiles(mi, rows_for(mi, std::max<int64_t>(kPMinRows * plan.mats[mi].m,
                                                          class_tile(K_PFUSED, 1 | kThreeWaves, 2 * kTileElems))));
        if (!vec_done) vec_tiles(bk), vec_done = true;
        sink.end(l, L);
      }
      if (!eight.empty()) {
        l = sink.begin(K_PFUSED, 2 | kEightWaves);
        for (int32_t mi : eight)
          pstep_tiles(mi, rows_for(mi, std::max<int64_t>(kPMinRows * plan.mats[mi].m,
                                                          class_tile(K_PFUSED, 2 | kEightWaves, 4 * kTileElems))));
        if (!vec_done) vec_tiles(bk), vec_done = true;
        sink.end(l, L);
      }
      if (pmerge >= 2) {
        bool any = false;
        for (int32_t S = 2; S <= 5; ++S)
          if (class_of_p(S) == pmerge && !of_class(S).empty()) any = true;
        if (any) {
          l = sink.begin(K_PFUSED, pmerge);
          for (int32_t S = 2; S <= 5; ++S)
            if (class_of_p(S) == pmerge) pfused_tiles(S);
          if (!vec_done) vec_tiles(bk), vec_done = true;
          sink.end(l, L);
        }
      }
      if (!generic.empty()) {
        l = sink.begin(K_PROW, 0);
        for (int32_t mi : generic) row_tiles(mi, 1);
        if (!vec_done) vec_tiles(bk), vec_done = true;
        sink.end(l, L);
        if (list_ef) {
          l = sink.begin(K_EUPD, 1);
          for (int32_t mi : generic)
            row_tiles(mi, std::max<int64_t>(1, kSmallTileElems / plan.mats[mi].m));
          sink.end(l, L);
        }
      }
      if (!vec_done) {
        l = sink.begin(K_VEC, 1);
        vec_tiles(bk);
        sink.end(l, L);
      }
    }
    // -- Q-step (even t)
    {
      std::vector<Launch>& L = bk.compress[0];
      bool vec_done = bk.vecs.empty();
      Launch l = sink.begin(K_APPLY, 0);
      apply_tiles(generic, false);
      sink.end(l, L);
      auto qtiles = [&](int32_t mi) {
        const MatDesc& d = plan.mats[mi];
        const int32_t ncb = static_cast<int32_t>(cdiv(d.m, d.q_cb));
        for (int32_t c = 0; c < d.q_chunks; ++c)
          for (int32_t cb = 0; cb < ncb; ++cb) plan.tiles.push_back(Tile{T_QTILE, mi, c, cb});
      };
      for (int32_t variant : {4 | kQFused, 4, 1}) {
        l = sink.begin(K_QSTEP, variant);
        bool any = false;
        if (variant & kQFused) {  // the small and narrow-row matrices ride in the fused launch
          small_tiles();
          for (int32_t mi : narrow) qtiles(mi);
          any = !small.empty() || !narrow.empty();
        }
        const std::vector<int32_t>& set = (variant & kQFused) ? fast : generic;
        if (variant & kQFused) {  // the three- and eight-wave P-step's matrices too
          for (int32_t mi : three) qtiles(mi), any = true;
          for (int32_t mi : eight) qtiles(mi), any = true;
        }
        for (int32_t mi : set) {
          if (!(variant & kQFused) && plan.mats[mi].q_cb != 4 * 64 * variant) continue;
          qtiles(mi);
          any = true;
        }
        if (any && !vec_done) vec_tiles(bk), vec_done = true;
        sink.end(l, L);
      }
      qfin_launch(bk, L, false);
      if (!vec_done) {
        l = sink.begin(K_VEC, 0);
        vec_tiles(bk);
        sink.end(l, L);
      }
    }
    // -- decompress (both parities): factor tiles first, then rows, then vectors
    for (int32_t par = 0; par < 2; ++par) {
      std::vector<Launch>& L = bk.decompress[par];
      const bool q = par == 0;
      bool extra_done = false;
      auto extra = [&]() {
        if (extra_done) return;
        for (int32_t mi : bk.mats) fact_tiles(mi, q);
        vec_tiles(bk);
        extra_done = true;
      };
      if (!fast.empty() || !narrow.empty() || !small.empty() || !three.empty() || !eight.empty()) {
        Launch l = sink.begin(K_RECON4, 0);
        extra();
        small_tiles();
        for (int32_t v : narrow_vars)
          for (int32_t mi : of_narrow(v)) row_tiles(mi, narrow_rows(mi, class_tile(K_RNARROW, v, kTileElems)));
        for (int32_t mi : fast) recon4_tiles(mi);
        for (int32_t mi : three) recon4_tiles(mi);
        for (int32_t mi : eight) recon4_tiles(mi);
        sink.end(l, L);
      }
      for (int32_t vw : {4, 1}) {
        Launch l = sink.begin(K_RECON, vw);
        bool any = false;
        for (int32_t mi : generic)
          if ((vw == 4) == is_vec4(mi)) any = true;
        if (any || vw == 1) extra();
        for (int32_t mi : generic)
          if ((vw == 4) == is_vec4(mi))
            row_tiles(mi, std::max<int64_t>(1, 2 * kSmallTileElems / plan.mats[mi].m));
        sink.end(l, L);
      }
      {
        Launch l = sink.begin(K_CHOL, 0);
        for (int32_t mi : bk.mats) chol_tiles(mi, q);
        sink.end(l, L);
      }
    }
    emat_launch(bk);
  }
  // ---- no reuse: before each compress the reused factor is drawn anew (K_DRAW) and its W formed
  // (factor tiles from its slot, then the Gram finish); [1]: P-steps draw Q, [0]: Q-steps draw P
  for (BucketPlan& bk : plan.buckets) {
    if (reuse) break;
    for (int32_t par = 0; par < 2; ++par) {
      const bool q = par == 1;
      std::vector<Launch>& L = bk.draw[par];
      Launch l = sink.begin(K_DRAW, q ? 1 : 0);
      for (int32_t mi : bk.mats) {
        const int64_t rows = q ? plan.mats[mi].m : plan.mats[mi].n;
        for (int64_t s0 = 0; s0 < rows; s0 += kDrawRows)
          plan.tiles.push_back(Tile{T_ROWS, mi, static_cast<int32_t>(s0),
                                    static_cast<int32_t>(std::min<int64_t>(kDrawRows, rows - s0))});
      }
      sink.end(l, L);
      l = sink.begin(K_FACT, q ? 1 : 0);
      for (int32_t mi : bk.mats) fact_tiles(mi, q);
      sink.end(l, L);
      chol_launches(bk.mats, q, L);
    }
  }
  // ---- Power-SGD: the first half writes M' = M + E (raw vectors too) into the E arena and sets
  // W = I, then runs the P-step lists on it; the second half copies the all-reduced P into its slot
  // and forms its W, then runs the Q-step lists; decompress is the Q-step decompress
  for (BucketPlan& bk : plan.buckets) {
    if (!psgd) break;
    Launch l = sink.begin(K_IMAGE, 0);
    const int64_t ir = image_rows(rank);
    for (int32_t mi : bk.mats) {
      plan.tiles.push_back(Tile{T_FACT, mi, 0, 0});
      if (!ef) continue;
      const MatDesc& d = plan.mats[mi];
      const int64_t ncb = cdiv(d.m, kImageCols);
      for (int64_t r0 = 0; r0 < d.n; r0 += ir)
        for (int64_t cb = 0; cb < ncb; ++cb)
          plan.tiles.push_back(Tile{T_QTILE, mi, static_cast<int32_t>(r0),
                                    static_cast<int32_t>(cb | (std::min<int64_t>(ir, d.n - r0) << 16))});
    }
    if (ef) vec_tiles(bk);
    sink.end(l, bk.psgd_image);
    l = sink.begin(K_FACT, kFactFromBuffer);
    for (int32_t mi : bk.mats) fact_tiles(mi, false);
    sink.end(l, bk.psgd_fact);
    chol_launches(bk.mats, false, bk.psgd_fact);
  }
  {
    Launch l = sink.begin(K_FACT, 1);
    for (int32_t mi = 0; mi < static_cast<int32_t>(plan.mats.size()); ++mi) fact_tiles(mi, true);
    sink.end(l, plan.gram_init);
    std::vector<int32_t> all(plan.mats.size());
    for (int32_t mi = 0; mi < static_cast<int32_t>(plan.mats.size()); ++mi) all[mi] = mi;
    chol_launches(all, true, plan.gram_init);
  }

  // ---- launch families and algorithmic bytes (host-side profiling)
  auto tile_bytes = [&](const Launch& l, const Tile& t, bool odd) -> double {
    const double eb = list_ef ? 12.0 : 4.0;  // M read, E read, E written per compress element
    if (t.kind == T_VEC) return 8.0 * t.b;
    const MatDesc& d = plan.mats[t.idx];
    const double n = d.n, m = d.m, rr = double(r);
    if (t.kind == T_SMALL) {  // a whole small matrix: P-step, Q-step (with its finish), decompress
      if (l.kernel == K_PFUSED) return n * m * eb + n * rr * 8.0 + m * rr * 12.0;
      if (l.kernel == K_QSTEP) return n * m * eb + n * rr * 8.0 + m * rr * 8.0;
      return n * m * 4.0 + n * rr * 4.0 + m * rr * 4.0;
    }
    switch (l.kernel) {
      case K_PFUSED: {  // strided tiles, or a narrow-row matrix's block of rows
        const double rows = t.kind == T_SROWS ? double(t.b >> 16) : double(t.b);
        return rows * m * eb + rows * rr * 8.0 + (t.a == 0 ? m * rr * 12.0 : 0.0);
      }
      case K_PROW:
        return m * (list_ef ? 8.0 : 4.0) + rr * 8.0 + (t.a == 0 ? m * rr * 12.0 : 0.0);
      case K_EUPD:
        return t.b * m * 4.0;
      case K_QSTEP: {
        const double rows = q_chunk_rows(d, t.a).rows;
        const double cols = std::min<double>(d.q_cb, m - double(t.b) * d.q_cb);
        return rows * cols * eb + (t.b == 0 ? rows * rr * 8.0 : 0.0);
      }
      case K_QFIN: {
        const double ne = qfin_entries(d.q_chunks), e0 = double(t.a) * ne;
        return 8.0 * std::max(0.0, std::min<double>(ne, m * rr - e0));
      }
      case K_RECON:
      case K_RECON4:
        if (t.kind == T_FACT) {
          const double rows = odd ? n : m;
          return std::min<double>(d.fact_rows, rows - double(t.a) * d.fact_rows) * rr * 8.0;
        }
        if (t.kind == T_SROWS) {
          const double rows = t.b >> 16, cols = std::min<double>(1024.0, m - 1024.0 * (t.b & 15));
          return rows * cols * 4.0 + rows * rr * 4.0 + (t.a == 0 ? cols * rr * 4.0 : 0.0);
        }
        return t.b * m * 4.0 + t.b * rr * 4.0 + (t.a == 0 ? m * rr * 4.0 : 0.0);
      case K_WPSTEP:
        return t.b * m * eb + t.b * rr * 8.0 + (t.a == 0 ? m * rr * 8.0 : 0.0);
      case K_WQSTEP: {
        const double r0 = double(t.a) * d.q_rows;
        const double rows = std::min<double>(d.q_rows, n - r0);
        const double cw = double(d.q_cb) * (r < kSplitRank ? kWideQWaves : 1);  // a tile's columns
        const double cols = std::min<double>(cw, m - double(t.b) * cw);
        return rows * cols * eb + (t.b == 0 ? rows * rr * 8.0 : 0.0);
      }
      case K_WFACT: {  // from kBlockedRank on a slice's rows are read and copied once, counted on its first part
        const double rows = odd ? n : m;
        if (t.a >> 16) return 0.0;
        return std::min<double>(d.fact_rows, rows - double(t.a & 0xffff) * d.fact_rows) * rr * 8.0;
      }
      case K_WRECON: {
        const double rows = std::min<double>(32.0, n - 32.0 * t.a);
        const double cols = std::min<double>(kWideRCols, m - double(kWideRCols) * t.b);
        return rows * cols * 4.0 + (t.b == 0 ? rows * rr * 4.0 : 0.0) + (t.a == 0 ? cols * rr * 4.0 : 0.0);
      }
      case K_APPLY:  // from kApplyMfmaRank on a tile covers one of apply_blocks(r) column blocks
        return (t.b & 0xffff) * rr * 8.0 / apply_blocks(static_cast<int32_t>(r));
      case K_FACT:
        if (t.a >> 16) return 0.0;
        return std::min<double>(d.fact_rows, (l.variant & 1 ? m : n) - double(t.a & 0xffff) * d.fact_rows) * rr *
               (l.variant & kFactFromBuffer ? 8.0 : 4.0);
      case K_EMAT:
        return t.b * m * 8.0;
      case K_GSUM:  // the slices' partials read, the sum written
        return (t.b + 1.0) * kGsumEntries * 8.0;
      case K_DRAW:
        return t.b * rr * 4.0;
      case K_IMAGE: {  // M read, E read, M' written
        if (t.kind != T_QTILE) return 0.0;
        const double cols = std::min<double>(kImageCols, m - double(t.b & 0xffff) * kImageCols);
        return double(t.b >> 16) * cols * 12.0;
      }
      default:
        return 0.0;
    }
  };
  auto family_of = [](int32_t kernel, bool odd) -> int32_t {
    switch (kernel) {
      case K_PFUSED: case K_PROW: case K_EUPD: case K_WPSTEP: case K_IMAGE:
        return 1;  // ACP_KERNEL_P_STEP
      case K_QSTEP: case K_WQSTEP:
        return 2;  // ACP_KERNEL_Q_STEP
      case K_QFIN: return 3;  // ACP_KERNEL_Q_FINISH
      case K_RECON: case K_RECON4: case K_WRECON:
        return 4;  // ACP_KERNEL_RECONSTRUCT
      case K_WFACT: return 5;                                              // ACP_KERNEL_ORTH
      case K_APPLY: case K_FACT: case K_CHOL: case K_GSUM: case K_DRAW: return 5;  // ACP_KERNEL_ORTH
      default: return 0;  // K_VEC (raw-vector launches of their own) and K_EMAT: no family
    }
  };
  auto annotate = [&](std::vector<Launch>& list, bool odd) {
    for (Launch& l : list) {
      l.family = family_of(l.kernel, odd);
      l.alg_bytes = 0.0;
      for (int32_t i = 0; i < l.ntiles; ++i) l.alg_bytes += tile_bytes(l, plan.tiles[l.tile_off + i], odd);
    }
  };
  for (BucketPlan& bk : plan.buckets) {
    annotate(bk.compress[0], false);
    annotate(bk.compress[1], true);
    annotate(bk.decompress[0], false);
    annotate(bk.decompress[1], true);
    annotate(bk.emat, false);
    annotate(bk.draw[0], false);
    annotate(bk.draw[1], true);
    annotate(bk.psgd_image, true);
    annotate(bk.psgd_fact, false);
  }
  annotate(plan.gram_init, false);

  // ---- launches over whole groups of buckets: every bucket's launches of one kind merged into
  // one, in the dependency order the per-bucket lists already follow
  auto order_of = [](const Launch& l) -> int32_t {
    switch (l.kernel) {
      case K_DRAW: case K_IMAGE: return -3;
      case K_FACT: return -2;
      case K_APPLY: return 0;
      case K_PFUSED: return (l.variant & kEightWaves) ? 8 : (l.variant & kThreeWaves) ? 7 : 1 + l.variant;  // 2..8
      case K_PROW: return 10;
      case K_EUPD: return 11;
      case K_WPSTEP: return 12;
      case K_WQSTEP: return 22;
      case K_WRECON: return 40;
      case K_WFACT: return 41;
      case K_QSTEP: return (l.variant & kQFused) ? 20 : (l.variant == 4 ? 21 : 22);
      case K_QFIN: return 23;
      case K_RECON4: return 31;
      case K_RECON: return l.variant == 4 ? 40 : 41;
      case K_GSUM: return 42;
      case K_CHOL: return 43;
      case K_VEC: return 50;
      default: return 60;
    }
  };
  auto merge = [&](int32_t b0, int32_t b1, auto get, bool odd) {
    std::vector<Launch> all;
    for (int32_t b = b0; b < b1; ++b)
      for (const Launch& l : get(plan.buckets[b])) all.push_back(l);
    // sorted by kind, then variant: every (kernel, variant) of the group becomes one launch
    std::stable_sort(all.begin(), all.end(), [&](const Launch& x, const Launch& y) {
      return order_of(x) != order_of(y) ? order_of(x) < order_of(y) : x.variant < y.variant;
    });
    std::vector<Launch> out;
    for (size_t i = 0; i < all.size();) {
      size_t j = i;
      Launch m = all[i];
      m.tile_off = static_cast<int64_t>(plan.tiles.size());
      m.ntiles = 0;
      m.alg_bytes = 0.0;
      // the launch's tiles, longest first so that no long tile starts last; factor tiles
      // (short in bytes but a serial Gram / Cholesky) lead
      std::vector<std::pair<double, Tile>> ts;
      while (j < all.size() && all[j].kernel == all[i].kernel && all[j].variant == all[i].variant) {
        for (int32_t k = 0; k < all[j].ntiles; ++k) {
          const Tile tc = plan.tiles[all[j].tile_off + k];
          const double w = tc.kind == T_FACT ? 1e30 : tile_bytes(all[j], tc, odd);
          ts.emplace_back(w, tc);
        }
        m.ntiles += all[j].ntiles;
        m.alg_bytes += all[j].alg_bytes;
        ++j;
      }
      std::stable_sort(ts.begin(), ts.end(),
                       [](const std::pair<double, Tile>& x, const std::pair<double, Tile>& y) {
                         return x.first > y.first;
                       });
      for (const auto& p : ts) plan.tiles.push_back(p.second);
      out.push_back(m);
      i = j;
    }
    return out;
  };
  {
    const int32_t nb = static_cast<int32_t>(plan.buckets.size());
    for (int32_t b0 = 0; b0 < nb; b0 += kMaxGroup) {
      const int32_t b1 = std::min(nb, b0 + kMaxGroup);
      std::array<std::vector<Launch>, 2> gc, gd;
      for (int32_t par = 0; par < 2; ++par) {
        gc[par] = merge(b0, b1, [par](const BucketPlan& bk) -> const std::vector<Launch>& { return bk.compress[par]; }, par == 1);
        gd[par] = merge(b0, b1, [par](const BucketPlan& bk) -> const std::vector<Launch>& { return bk.decompress[par]; }, par == 1);
      }
      plan.group_compress.push_back(gc);
      plan.group_decompress.push_back(gd);
      std::array<std::vector<Launch>, 2> gw;
      for (int32_t par = 0; par < 2; ++par)
        gw[par] = merge(b0, b1, [par](const BucketPlan& bk) -> const std::vector<Launch>& { return bk.draw[par]; }, par == 1);
      plan.group_draw.push_back(gw);
      plan.group_psgd_image.push_back(
          merge(b0, b1, [](const BucketPlan& bk) -> const std::vector<Launch>& { return bk.psgd_image; }, true));
      plan.group_psgd_fact.push_back(
          merge(b0, b1, [](const BucketPlan& bk) -> const std::vector<Launch>& { return bk.psgd_fact; }, false));
    }
  }

  // ---- region offsets (bytes)
  auto a256 = [](int64_t x) { return align_up(x, 256); };
  plan.e_floats = e_floats;
  plan.fac_floats = fac_floats;
  plan.w_doubles = static_cast<int64_t>(plan.mats.size()) * r * r;
  plan.gpart_doubles = gpart;
  plan.qpart_floats = qpart;
  int64_t off = 0;
  plan.off_e = off;     off = a256(off + e_floats * 4);
  plan.off_fac = off;   off = a256(off + fac_floats * 4);
  plan.off_w = off;     off = a256(off + plan.w_doubles * 8);
  plan.off_gpart = off; off = a256(off + gpart * 8);
  plan.off_qpart = off; off = a256(off + qpart * 4);
  plan.off_mats = off;  off = a256(off + static_cast<int64_t>(plan.mats.size() * sizeof(MatDesc)));
  plan.off_vecs = off;  off = a256(off + static_cast<int64_t>(plan.vecs.size() * sizeof(VecDesc)));
  plan.off_tiles = off; off = a256(off + static_cast<int64_t>(plan.tiles.size() * sizeof(Tile)));
  plan.total_bytes = std::max<int64_t>(off, 256);
  return "";
}

}  // namespace acp
