// Host-side planner of the ACP-SGD library: layout, initial factors, state regions and the
// launch tables of every bucket and phase.  HIP-free: it builds and runs without a GPU.
#pragma once

#include <cstdint>
#include <array>
#include <string>
#include <vector>

#include "acp_internal.hpp"

namespace acp {

struct TensorPlan {
  std::vector<int64_t> shape;
  int64_t numel = 0;
  bool compressed = false;
  int64_t n = 0, m = 1;     // matrix shape (numel x 1 for passthrough tensors)
  int32_t bucket = -1;      // bucket index
  int32_t pos = -1;         // position inside the bucket
  int32_t mat = -1;         // index into Plan::mats (compressed) or -1
  int32_t vec = -1;         // index into Plan::vecs (passthrough) or -1
};

struct BucketPlan {
  std::vector<int32_t> tids;
  std::vector<int64_t> grad_off, fac_off_p, fac_off_q;
  int64_t grad_elems = 0, fac_elems_p = 0, fac_elems_q = 0;
  int64_t e_base = 0;                 // E arena offset of the bucket (floats)
  int64_t qpart_base = 0;             // first Q-step partial of the bucket's matrices (floats)
  int64_t qpart_floats = 0;           // Q-step partials of the bucket's matrices (floats)
  std::vector<int32_t> mats, vecs;    // members by kind
  std::vector<Launch> compress[2];    // [0] even step (Q-step), [1] odd step (P-step)
  std::vector<Launch> decompress[2];
  std::vector<Launch> emat;
  std::vector<Launch> draw[2];        // no reuse: the fresh reused factor and its W, before compress
  std::vector<Launch> psgd_image;     // Power-SGD, first half: M' into the E arena, W = I
  std::vector<Launch> psgd_fact;      // Power-SGD, second half: the all-reduced P into its slot, W
};

struct Plan {
  int32_t rank = 0;
  int64_t cap_bytes = 0;
  bool ef = true;
  bool reuse = true;   // reuse the previous factor (else draw it anew every step)
  bool psgd = false;   // Power-SGD (Algorithm 1) instead of ACP-SGD
  std::vector<TensorPlan> tensors;
  std::vector<BucketPlan> buckets;
  std::vector<MatDesc> mats;
  std::vector<VecDesc> vecs;
  std::vector<Tile> tiles;
  std::vector<Launch> gram_init;     // W of every matrix's Q slot (after bind / restore)
  // launches covering whole groups of kMaxGroup buckets (the *_all entry points):
  // [group][parity] -> launches
  std::vector<std::array<std::vector<Launch>, 2>> group_compress, group_decompress, group_draw;
  std::vector<std::vector<Launch>> group_psgd_image, group_psgd_fact;

  // device state regions (byte offsets from the block base)
  int64_t off_e = 0, off_fac = 0, off_w = 0, off_gpart = 0, off_qpart = 0;
  int64_t off_mats = 0, off_vecs = 0, off_tiles = 0, total_bytes = 0;
  int64_t e_floats = 0, fac_floats = 0, w_doubles = 0, gpart_doubles = 0, qpart_floats = 0;
};

// Builds the plan; returns "" on success or an error text.
// reuse = false: ACP-SGD drawing the reused factor anew every step; psgd: Power-SGD (needs reuse).
std::string build_plan(Plan& plan, int32_t num_tensors, const int32_t* ndims, const int64_t* dims,
                       int32_t rank, int64_t cap_bytes, bool ef, bool reuse = true, bool psgd = false);

// Initial factor (f = 0: P_0, n x r; f = 1: Q_0, m x r) of tensor `tid`, row-major fp32.
void draw_init_factor(uint64_t seed, int32_t tid, int32_t f, int64_t count, float* out);

// SplitMix64 output finaliser.
uint64_t splitmix64_mix(uint64_t z);

}  // namespace acp
