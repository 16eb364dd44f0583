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

namespace acp {

namespace {

constexpr int64_t kTileElems = 16384;   // gradient elements per streaming tile
constexpr int64_t kVecChunk = 4096;     // raw-vector elements per copy tile
constexpr int64_t kApplyRows = 256;     // factor rows per orthogonalisation tile
constexpr int64_t kSlotAlign = 64;      // floats (256 bytes)

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
int64_t align_up(int64_t x, int64_t a) { return cdiv(x, a) * a; }

bool rank_supported(int32_t r) { return r == 1 || r == 2 || r == 4 || r == 8 || r == 16 || r == 32; }

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
                       int32_t rank, int64_t cap_bytes, bool ef) {
  if (num_tensors <= 0) return "num_tensors must be positive";
  if (!ndims || !dims) return "ndims and dims must not be NULL";
  if (!rank_supported(rank)) return "rank must be one of 1, 2, 4, 8, 16, 32";
  if (cap_bytes <= 0) return "bucket_cap_bytes must be positive";
  plan = Plan{};
  plan.rank = rank;
  plan.cap_bytes = cap_bytes;
  plan.ef = ef;
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
      if (m < (int64_t(1) << 31) && r < std::min(n, m)) {
        t.compressed = true;
        t.n = n;
        t.m = m;
      }
    }
    if (!t.compressed) {
      t.n = numel;
      t.m = 1;
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

  // ---- per-tensor device descriptors and state regions
  int64_t e_floats = 0, fac_floats = 0, gpart = 0, qpart = 0, nctr = 0;
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
      const int64_t np = align_up(t.n * r, kSlotAlign), mp = align_up(t.m * r, kSlotAlign);
      d.p_slot = fac_floats;
      d.ph_slot = fac_floats + np;
      d.q_slot = fac_floats + 2 * np;
      d.qh_slot = fac_floats + 2 * np + mp;
      d.ql_slot = fac_floats + 2 * np + 2 * mp;
      fac_floats += 2 * np + 3 * mp;
      const bool vec4 = (t.m % 4 == 0) && (d.grad_off % 4 == 0);
      const int64_t cpt = (vec4 && r <= 8) ? 4 : 1;
      d.q_cb = static_cast<int32_t>(64 * cpt);
      d.q_rows = static_cast<int32_t>(align_up(std::max<int64_t>(32, cdiv(t.n, 64)), 4));
      d.q_chunks = static_cast<int32_t>(cdiv(t.n, d.q_rows));
      const int64_t ncb = cdiv(t.m, d.q_cb);
      d.qpart = qpart;
      qpart += align_up(int64_t(d.q_chunks) * ncb * d.q_cb * r, kSlotAlign);
      d.fact_rows = r <= 8 ? 1024 : 256;
      const int64_t gsl = std::max(cdiv(t.n, d.fact_rows), cdiv(t.m, d.fact_rows));
      d.gpart = gpart;
      gpart += gsl * r * r;
      d.w_slot = static_cast<int64_t>(plan.mats.size()) * r * r;
      d.ctr_gram = static_cast<int32_t>(nctr++);
      d.ctr_q = static_cast<int32_t>(nctr);
      nctr += ncb;
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
  auto apply_tiles = [&](const BucketPlan& bk, bool q) {
    for (int32_t mi : bk.mats) {
      const int64_t rows = q ? plan.mats[mi].m : plan.mats[mi].n;
      for (int64_t s = 0; s < rows; s += kApplyRows)
        plan.tiles.push_back(Tile{T_ROWS, mi, static_cast<int32_t>(s),
                                  static_cast<int32_t>(std::min(kApplyRows, rows - s))});
    }
  };
  auto fact_tiles = [&](int32_t mi, bool q) {
    const MatDesc& d = plan.mats[mi];
    const int64_t rows = q ? d.m : d.n;
    const int32_t nsl = static_cast<int32_t>(cdiv(rows, d.fact_rows));
    for (int32_t s = 0; s < nsl; ++s) plan.tiles.push_back(Tile{T_FACT, mi, s, nsl});
  };
  auto row_tiles = [&](int32_t mi, int64_t rows_per_tile) {
    const MatDesc& d = plan.mats[mi];
    for (int64_t s = 0; s < d.n; s += rows_per_tile)
      plan.tiles.push_back(Tile{T_ROWS, mi, static_cast<int32_t>(s),
                                static_cast<int32_t>(std::min<int64_t>(rows_per_tile, d.n - s))});
  };
  auto is_vec4 = [&](int32_t mi) {
    const MatDesc& d = plan.mats[mi];
    return d.m % 4 == 0 && d.grad_off % 4 == 0;
  };

  for (BucketPlan& bk : plan.buckets) {
    // -- P-step (odd t)
    {
      std::vector<Launch>& L = bk.compress[1];
      Launch l = sink.begin(K_APPLY, 1);
      apply_tiles(bk, true);
      sink.end(l, L);
      std::vector<int32_t> fused, generic;
      int32_t S = 1;
      for (int32_t mi : bk.mats) {
        const int64_t m4 = plan.mats[mi].m / 4;
        if (r == 4 && is_vec4(mi) && cdiv(m4, 256) <= 5) {
          fused.push_back(mi);
          S = std::max<int32_t>(S, static_cast<int32_t>(cdiv(m4, 256)));
        } else {
          generic.push_back(mi);
        }
      }
      bool vec_done = bk.vecs.empty();
      if (!fused.empty()) {
        l = sink.begin(K_PFUSED, S);
        for (int32_t mi : fused) {
          MatDesc& d = plan.mats[mi];
          d.wpr = static_cast<int32_t>(cdiv(d.m / 4, 64 * int64_t(S)));
          const int64_t rpr = 4 / d.wpr;
          const int64_t rows = rpr * std::max<int64_t>(1, kTileElems / (int64_t(d.m) * rpr));
          row_tiles(mi, rows);
        }
        if (!vec_done) vec_tiles(bk), vec_done = true;
        sink.end(l, L);
      }
      if (!generic.empty()) {
        l = sink.begin(K_PROW, 0);
        for (int32_t mi : generic) row_tiles(mi, 1);
        if (!vec_done) vec_tiles(bk), vec_done = true;
        sink.end(l, L);
        if (ef) {
          l = sink.begin(K_EUPD, 1);
          for (int32_t mi : generic)
            row_tiles(mi, std::max<int64_t>(1, kTileElems / plan.mats[mi].m));
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
      Launch l = sink.begin(K_APPLY, 0);
      apply_tiles(bk, false);
      sink.end(l, L);
      bool vec_done = bk.vecs.empty();
      for (int32_t cpt : {4, 1}) {
        l = sink.begin(K_QSTEP, cpt);
        bool any = false;
        for (int32_t mi : bk.mats) {
          const MatDesc& d = plan.mats[mi];
          if (d.q_cb != 64 * cpt) continue;
          any = true;
          const int32_t ncb = static_cast<int32_t>(cdiv(d.m, d.q_cb));
          for (int32_t c = 0; c < d.q_chunks; ++c)
            for (int32_t cb = 0; cb < ncb; ++cb) plan.tiles.push_back(Tile{T_QTILE, mi, c, cb});
        }
        if (any && !vec_done) vec_tiles(bk), vec_done = true;
        sink.end(l, L);
      }
      if (!vec_done) {
        l = sink.begin(K_VEC, 0);
        vec_tiles(bk);
        sink.end(l, L);
      }
    }
    // -- decompress (both parities) and E export
    for (int32_t par = 0; par < 2; ++par) {
      std::vector<Launch>& L = bk.decompress[par];
      bool extra_done = false;
      for (int32_t vw : {4, 1}) {
        Launch l = sink.begin(K_RECON, vw);
        for (int32_t mi : bk.mats)
          if ((vw == 4) == is_vec4(mi))
            row_tiles(mi, std::max<int64_t>(1, kTileElems / plan.mats[mi].m));
        const bool any = static_cast<int64_t>(plan.tiles.size()) > l.tile_off;
        if ((any || vw == 1) && !extra_done) {
          for (int32_t mi : bk.mats) fact_tiles(mi, par == 0);
          vec_tiles(bk);
          extra_done = true;
        }
        sink.end(l, L);
      }
    }
    {
      Launch l = sink.begin(K_EMAT, 1);
      for (int32_t mi : bk.mats) row_tiles(mi, std::max<int64_t>(1, kTileElems / plan.mats[mi].m));
      sink.end(l, bk.emat);
    }
  }
  {
    Launch l = sink.begin(K_GRAM, 1);
    for (int32_t mi = 0; mi < static_cast<int32_t>(plan.mats.size()); ++mi) fact_tiles(mi, true);
    sink.end(l, plan.gram_init);
  }

  // ---- region offsets (bytes)
  auto a256 = [](int64_t x) { return align_up(x, 256); };
  plan.e_floats = e_floats;
  plan.fac_floats = fac_floats;
  plan.w_doubles = static_cast<int64_t>(plan.mats.size()) * r * r;
  plan.gpart_doubles = gpart;
  plan.qpart_floats = qpart;
  plan.n_ctr = nctr;
  int64_t off = 0;
  plan.off_e = off;     off = a256(off + e_floats * 4);
  plan.off_fac = off;   off = a256(off + fac_floats * 4);
  plan.off_w = off;     off = a256(off + plan.w_doubles * 8);
  plan.off_gpart = off; off = a256(off + gpart * 8);
  plan.off_qpart = off; off = a256(off + qpart * 4);
  plan.off_ctr = off;   off = a256(off + nctr * 4);
  plan.off_mats = off;  off = a256(off + static_cast<int64_t>(plan.mats.size() * sizeof(MatDesc)));
  plan.off_vecs = off;  off = a256(off + static_cast<int64_t>(plan.vecs.size() * sizeof(VecDesc)));
  plan.off_tiles = off; off = a256(off + static_cast<int64_t>(plan.tiles.size() * sizeof(Tile)));
  plan.total_bytes = std::max<int64_t>(off, 256);
  return "";
}

}  // namespace acp
