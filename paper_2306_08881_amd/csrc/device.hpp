// Device helpers shared by the gfx950 kernel files: lane and buffer primitives, DPP wave
// sums, bucket buffers of a launch, raw-vector tiles and the Gram/Cholesky orthogonalisation
// tiles (arXiv 2306.08881, Algorithm 2: the orthogonalisation of the reused factor).
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

#include "acp_internal.hpp"

namespace acp {
namespace {

__device__ inline int tid() { return static_cast<int>(threadIdx.x); }

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ inline double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ inline float4 wave_sum(float4 v) {
  v.x = wave_sum(v.x);
  v.y = wave_sum(v.y);
  v.z = wave_sum(v.z);
  v.w = wave_sum(v.w);
  return v;
}

__device__ inline float dot4(const float4& a, const float4& b) {
  return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w;
}

__device__ inline float4 operator+(const float4& a, const float4& b) {
  return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

__device__ inline float4 scale4(const float4& a, float s) {
  return make_float4(a.x * s, a.y * s, a.z * s, a.w * s);
}

__device__ inline float4 fma4(float s, const float4& v, const float4& acc) {
  return make_float4(fmaf(s, v.x, acc.x), fmaf(s, v.y, acc.y), fmaf(s, v.z, acc.z),
                     fmaf(s, v.w, acc.w));
}

__device__ inline float4 zero4() { return make_float4(0.f, 0.f, 0.f, 0.f); }

// Streaming accesses: data read or written exactly once per step.
typedef float v4f __attribute__((ext_vector_type(4)));
__device__ inline float4 ld_stream(const float4* p) {
  const v4f v = __builtin_nontemporal_load(reinterpret_cast<const v4f*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ inline void st_stream(float4* p, const float4& v) {
  const v4f w = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(w, reinterpret_cast<v4f*>(p));
}

// Tile-relative buffer accesses.  A buffer resource spans one tile from its first element;
// a load past num_records returns zero and a store past it is dropped, so lanes and rows that
// fall outside the tile need no branch: they take the offset kOut (or any offset past the
// extent).  Branch-free loads and stores let the compiler count outstanding memory operations
// exactly, so stores stay in flight while the next rows' loads are waited for.  Every extent
// and in-tile offset is below 2^30, so kOut plus an offset does not wrap.
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr uint32_t kOut = 0x80000000u;
constexpr int kAuxNT = 2;  // cache policy: nontemporal (streamed once)

__device__ inline Rsrc tile_rsrc(const float* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), 0, static_cast<int>(bytes),
                                           0x00020000);
}
// The buffer builtins move raw 32-bit words (unsigned int); values cross them bit-cast.
typedef unsigned int v4u __attribute__((ext_vector_type(4)));
__device__ inline float4 bld4_nt(Rsrc r, uint32_t off) {
  const v4f v = __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kAuxNT));
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ inline float bld1_nt(Rsrc r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kAuxNT));
}
__device__ inline void bst4_nt(Rsrc r, uint32_t off, const float4& v) {
  const v4f w = {v.x, v.y, v.z, v.w};
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, w), r, off, 0, kAuxNT);
}
__device__ inline void bst4(Rsrc r, uint32_t off, const float4& v) {
  const v4f w = {v.x, v.y, v.z, v.w};
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, w), r, off, 0, 0);
}
__device__ inline float4 bld4(Rsrc r, uint32_t off) {
  const v4f v = __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ inline float bld1(Rsrc r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ inline void bst1(Rsrc r, uint32_t off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned int, v), r, off, 0, 0);
}
__device__ inline void bst1_nt(Rsrc r, uint32_t off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned int, v), r, off, 0, kAuxNT);
}

// Sum over the 64 lanes with DPP: quad butterflies, half-row and row mirrors give every lane
// its 16-lane row sum; the four row sums are then read out and added in row order.  Every lane
// gets the same bits.
template <int CTRL>
__device__ inline float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                               0xF, 0xF, false));
}
__device__ inline float wave_sum_dpp(float v) {
  v += dpp<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp<0x141>(v);  // row_half_mirror
  v += dpp<0x140>(v);  // row_mirror
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return ((r0 + r1) + r2) + r3;
}
__device__ inline float4 wave_sum_dpp(float4 v) {
  return make_float4(wave_sum_dpp(v.x), wave_sum_dpp(v.y), wave_sum_dpp(v.z), wave_sum_dpp(v.w));
}

// x W for one row of a rank-4 factor (W upper triangular, fp64, row-major), rounded to fp32.
__device__ inline float4 apply_w4(const float4& x, const double* W) {
  const double x0 = x.x, x1 = x.y, x2 = x.z, x3 = x.w;
  const double y0 = x0 * W[0];
  const double y1 = fma(x0, W[1], x1 * W[5]);
  const double y2 = fma(x0, W[2], fma(x1, W[6], x2 * W[10]));
  const double y3 = fma(x0, W[3], fma(x1, W[7], fma(x2, W[11], x3 * W[15])));
  return make_float4(static_cast<float>(y0), static_cast<float>(y1), static_cast<float>(y2),
                     static_cast<float>(y3));
}

// Buffers of a bucket in this launch's group.
__device__ inline const float* src_of(const KArgs& a, int32_t b) { return a.src[b - a.base]; }
__device__ inline float* dst_of(const KArgs& a, int32_t b) { return a.dst[b - a.base]; }
__device__ inline bool deferred_of(const KArgs& a, int32_t b) {
  return ((a.deferred >> (b - a.base)) & 1ull) != 0;
}
__device__ inline bool deferred_p_of(const KArgs& a, int32_t b) {
  return ((a.deferred_p >> (b - a.base)) & 1ull) != 0;
}

// Raw vectors: pack the gradient into the factor buffer (compress) or unpack the aggregated
// sum / p into the output bucket (decompress).
__device__ void vec_tile(const KArgs& a, const Tile& t, bool compress) {
  const VecDesc v = a.vecs[t.idx];
  const int64_t foff = a.parity ? v.fac_off_p : v.fac_off_q;
  const float* src = src_of(a, v.bucket);
  float* dst = dst_of(a, v.bucket);
  for (int i = tid(); i < t.b; i += static_cast<int>(blockDim.x)) {  // launches of 3 or 4 waves
    const int64_t k = static_cast<int64_t>(t.a) + i;
    if (compress)
      dst[foff + k] = src[v.grad_off + k];
    else
      dst[v.grad_off + k] = src[foff + k] * a.inv_p;
  }
}

// ---------------------------------------------------------------------------------------
// Orthogonalisation, Gram/Cholesky form.  For a factor X (k x r) the Gram-Schmidt factor is
// orth(X) = X W with W = R^-1 and G = X^T X = R^T R (R upper triangular, positive diagonal):
// the same columns as Gram-Schmidt in exact arithmetic.  G is accumulated in fp64 from fp32
// products (exact) and factored in fp64.  A column j is dropped (its column of W is zero) when
// G_jj = 0 or its residual d_j = G_jj - sum_{i<j} R_ij^2 is at most tau^2 G_jj, i.e. when the
// residual norm is at most tau times the column norm.

typedef double v4d __attribute__((ext_vector_type(4)));
template <int RK, bool DIAG, int NB = 4>
__device__ void gram_band(const float* X, int64_t r0, int64_t r1, float* copy, int I, int J, int nw, int w,
                          v4d (&acc)[NB][NB]);

// Gram of rows [r0, r1) of X (row-major, RK columns) into shared G (RK x RK), by the whole
// workgroup, in a fixed order; the rows are also copied to `copy` when it is set.
template <int RK>
__device__ void gram_rows(const float* X, int64_t r0, int64_t r1, double* G, float* copy) {
  static_assert(RK <= 8 || RK == 16 || RK == 32 || RK == 64, "from kBlockedRank on gram_blocked forms the Gram");
  if constexpr (RK <= 8) {
    constexpr int NT = RK * (RK + 1) / 2;
    constexpr int PER = 8;  // rows per thread per pass, loaded together
    double g[NT];
#pragma unroll
    for (int e = 0; e < NT; ++e) g[e] = 0.0;
    for (int64_t base = r0; base < r1; base += int64_t(kBlock) * PER) {
      float x[PER][RK];
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int64_t row = base + u * kBlock + tid();
#pragma unroll
        for (int k = 0; k < RK; ++k) x[u][k] = row < r1 ? X[row * RK + k] : 0.f;
      }
      if (copy) {
#pragma unroll
        for (int u = 0; u < PER; ++u) {
          const int64_t row = base + u * kBlock + tid();
          if (row < r1)
#pragma unroll
            for (int k = 0; k < RK; ++k) copy[row * RK + k] = x[u][k];
        }
      }
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        int e = 0;
#pragma unroll
        for (int i = 0; i < RK; ++i)
#pragma unroll
          for (int j = i; j < RK; ++j, ++e)
            g[e] = fma(static_cast<double>(x[u][i]), static_cast<double>(x[u][j]), g[e]);
      }
    }
    __shared__ double red[4][NT];
#pragma unroll
    for (int e = 0; e < NT; ++e) g[e] = wave_sum(g[e]);
    if ((tid() & 63) == 0)
#pragma unroll
      for (int e = 0; e < NT; ++e) red[tid() >> 6][e] = g[e];
    __syncthreads();
    if (tid() < NT) {
      const int e = tid();
      int i = 0, rem = e;
      while (rem >= RK - i) rem -= RK - i, ++i;
      const int j = i + rem;
      const double s = ((red[0][e] + red[1][e]) + red[2][e]) + red[3][e];
      G[i * RK + j] = s;
      G[j * RK + i] = s;
    }
    __syncthreads();
  } else if constexpr (RK == 16 || RK == 32 || RK == 64) {
    // on the fp64 matrix cores (gram_band, one band of all RK columns): the four waves take
    // interleaved steps of 16 rows, each forming the products a <= b of the band's 16-column
    // blocks; their sums are added into G in wave order, then the blocks a > b mirrored
    constexpr int NB = RK / 16;
    const int w = tid() / kWave, lane = tid() % kWave, i = lane % 16, k = lane / 16;
    v4d acc[NB][NB];
    gram_band<RK, true, NB>(X, r0, r1, copy, 0, 0, kBlock / kWave, w, acc);
    for (int q = 0; q < kBlock / kWave; ++q) {
      if (w == q)
#pragma unroll
        for (int a = 0; a < NB; ++a)
#pragma unroll
          for (int b = a; b < NB; ++b)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              double& g = G[(16 * a + 4 * v + k) * RK + 16 * b + i];
              g = q == 0 ? acc[a][b][v] : g + acc[a][b][v];
            }
      __syncthreads();
    }
    for (int e = tid(); e < RK * RK; e += kBlock) {
      const int r = e / RK, c = e % RK;
      if (r / 16 > c / 16) G[e] = G[c * RK + r];
    }
    __syncthreads();
  }
}

// The lane's double from lane `src` of the wave (src uniform).
__device__ inline double readlane_d(double v, int src) {
  const int2 h = __builtin_bit_cast(int2, v);
  return __builtin_bit_cast(double, make_int2(__builtin_amdgcn_readlane(h.x, src),
                                              __builtin_amdgcn_readlane(h.y, src)));
}

// Cholesky G = R^T R and W = R^-1 (dropped columns and rows zero), written to w_out.  G in
// shared; every thread of the workgroup calls this, the first wave does the work.  Right-looking,
// one column per lane: lane j keeps column j of the updated G in registers; at pivot k lane k's
// diagonal decides the drop, each lane forms its entry R[k][j] and stores it to row k of R in
// LDS, and the trailing update reads R[k][i] back from there (one broadcast read per two entries;
// the wave's LDS accesses take effect in order).  The subtractions come in the same order as in
// the left-looking form (pivot 0 first), so R is the same.  W = R^-1 on the kept columns, row by
// row (lane = row).
template <int RK>
__device__ __attribute__((always_inline)) void cholesky_w(const double* G, double* w_out) {
  __shared__ double R[RK * RK];
  __shared__ int drop[RK];
  if (tid() >= kWave) return;
  const int j = tid();
  const bool col = j < RK;
  double g[RK];
#pragma unroll
  for (int i = 0; i < RK; ++i) g[i] = col ? G[i * RK + j] : 0.0;
#pragma unroll
  for (int k = 0; k < RK; ++k) {
    const double gkk = G[k * RK + k];
    const double dk = readlane_d(g[k], k);
    const bool keep = gkk > 0.0 && dk > kTau * kTau * gkk;
    const double rkk = keep ? sqrt(dk) : 0.0;
    double rkj = 0.0;
    if (keep) rkj = j > k ? g[k] / rkk : (j == k ? rkk : 0.0);
    if (col) R[k * RK + j] = rkj;
    if (j == 0) drop[k] = keep ? 0 : 1;
    __builtin_amdgcn_wave_barrier();
    if (keep)
#pragma unroll
      for (int i = k + 1; i < RK; ++i) g[i] -= R[k * RK + i] * rkj;
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  // W = R^-1 by rows (lane = row a), right-looking: once W[a][i] is final it is subtracted
  // from every later column at once, so the loads of R and the products of a step are
  // independent and only the divisions form a chain.  W[a][c] = (delta_ac - sum over i < c of
  // R[i][c] W[a][i]) / R[c][c], the sum in increasing i (the terms i < a are zero); zero for a
  // dropped pivot c or c < a.
  const int arow = j;
  if (arow < RK) {
    double acc[RK];
#pragma unroll
    for (int c = 0; c < RK; ++c) acc[c] = (arow == c) ? 1.0 : 0.0;
#pragma unroll
    for (int i = 0; i < RK; ++i) {
      asm volatile("" ::: "memory");  // this step's loads of R only (the registers stay few)
      // no branch: a dropped pivot divides by one and is then discarded
      const bool use = drop[i] == 0 && arow <= i;
      const double q = acc[i] / (use ? R[i * RK + i] : 1.0);
      const double wi = use ? q : 0.0;
      acc[i] = wi;
#pragma unroll
      for (int c = i + 1; c < RK; ++c) acc[c] -= R[i * RK + c] * wi;
    }
#pragma unroll
    for (int c = 0; c < RK; ++c) w_out[arow * RK + c] = acc[c];
  }
}

// Band block X_I^T X_J of rows [r0, r1) of X (row-major, RK columns; 64-column bands I <= J)
// into acc, on the fp64 matrix cores: 4 x 4 products of 16 x 16 (v_mfma_f64_16x16x4f64, four rows
// of X each; operand entry [i][k] on lane i + 16 k, result entry [4 v + l / 16][l % 16] in item v
// of lane l), product (a, b) for the columns 16 a ... and 16 b ... of the two bands; a diagonal
// block (DIAG) skips its products a > b, whose entries lie below the diagonal.  The rows go in
// steps of 16, of which the wave takes steps w, w + nw, ...; each product adds them in increasing
// groups of four, and the wave's next step is requested before the current one's products.  A
// diagonal block also copies its steps' rows of the band to `copy` when set.
template <int RK, bool DIAG, int NB>
__device__ void gram_band(const float* X, int64_t r0, int64_t r1, float* copy, int I, int J, int nw, int w,
                          v4d (&acc)[NB][NB]) {
  constexpr int G = 4;  // groups of four rows per step
  constexpr int BW = 16 * NB;  // band width (columns)
  const int lane = tid() % kWave, i = lane % 16, k = lane / 16;
  const float* xa = X + BW * I + i;
  const float* xb = X + BW * J + i;
#pragma unroll
  for (int a = 0; a < NB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[a][b] = v4d{0.0, 0.0, 0.0, 0.0};
  // rows past the slice read its last row (no branch around the loads, so the wait for a step's
  // rows leaves the next step's requests in flight); the A operand of those rows is zeroed
  auto row_of = [&](int64_t g0, int s) {
    const int64_t row = g0 + 4 * s + k;
    return row < r1 ? row : r1 - 1;
  };
  // two register buffers of G groups, filled and consumed in turn
  typedef float Buf[G][NB];
  auto fetch = [&](int64_t g0, Buf& ba, Buf& bb) {
#pragma unroll
    for (int s = 0; s < G; ++s) {
      const float* pa = xa + row_of(g0, s) * RK;
      const float* pb = xb + row_of(g0, s) * RK;
#pragma unroll
      for (int a = 0; a < NB; ++a) {
        ba[s][a] = pa[16 * a];
        if (!DIAG) bb[s][a] = pb[16 * a];
      }
    }
  };
  auto step = [&](int64_t g0, Buf& ba, Buf& bb) {
    // the conversions stay behind the other buffer's requests, issued just before
#pragma unroll
    for (int s = 0; s < G; ++s)
#pragma unroll
      for (int a = 0; a < NB; ++a) {
        asm volatile("" : "+v"(ba[s][a]));
        if (!DIAG) asm volatile("" : "+v"(bb[s][a]));
      }
    // a row past the slice stores its clamped row's own values again
    if (DIAG && copy)
#pragma unroll
      for (int s = 0; s < G; ++s)
#pragma unroll
        for (int a = 0; a < NB; ++a) copy[row_of(g0, s) * RK + BW * I + 16 * a + i] = ba[s][a];
#pragma unroll
    for (int s = 0; s < G; ++s) {
      const bool in = g0 + 4 * s + k < r1;
      double xa4[NB], xb4[NB];
#pragma unroll
      for (int a = 0; a < NB; ++a) {
        xa4[a] = in ? static_cast<double>(ba[s][a]) : 0.0;
        xb4[a] = static_cast<double>(DIAG ? ba[s][a] : bb[s][a]);
      }
#pragma unroll
      for (int a = 0; a < NB; ++a)
#pragma unroll
        for (int b = 0; b < NB; ++b)
          if (!DIAG || a <= b) acc[a][b] = __builtin_amdgcn_mfma_f64_16x16x4f64(xa4[a], xb4[b], acc[a][b], 0, 0, 0);
    }
  };
  // steps of 4 G rows: this wave takes steps w, w + nw, ... of the slice
  const int64_t sd = 4 * G * nw;
  Buf a0, b0, a1, b1;
  fetch(r0 + 4 * G * w, a0, b0);
  for (int64_t g0 = r0 + 4 * G * w; g0 < r1; g0 += 2 * sd) {  // a second step past the slice adds zeros
    fetch(g0 + sd, a1, b1);
    step(g0, a0, b0);
    fetch(g0 + 2 * sd, a0, b0);
    step(g0 + sd, a1, b1);
  }
}

// Part `part` of the Gram of rows [r0, r1) of X (RK >= kBlockedRank columns) into `out` (RK x RK
// doubles, global memory): G is symmetric, so only its band blocks with I <= J are formed
// (gram_band), numbered row by row; wave w of part p takes block 4 p + w over all the rows.
// K_GSUM mirrors the entries of the 4 x 4 blocks above the diagonal.
template <int RK>
__device__ void gram_blocked(const float* X, int64_t r0, int64_t r1, double* out, float* copy, int part) {
  constexpr int NB = RK / 64, NP = NB * (NB + 1) / 2;
  static_assert(gram_parts(RK) * (kBlock / kWave) >= NP, "every band block needs a wave");
  const int pr = part * (kBlock / kWave) + tid() / kWave;
  if (pr >= NP) return;
  int I = 0, rem = pr;
  while (rem >= NB - I) rem -= NB - I, ++I;
  const int J = I + rem, lane = tid() % kWave, i = lane % 16, k = lane / 16;
  v4d acc[4][4];
  if (rem == 0)
    gram_band<RK, true>(X, r0, r1, copy, I, I, 1, 0, acc);
  else
    gram_band<RK, false>(X, r0, r1, copy, I, J, 1, 0, acc);
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b)
      if (rem != 0 || a <= b)
#pragma unroll
        for (int v = 0; v < 4; ++v) out[(64 * I + 16 * a + 4 * v + k) * RK + 64 * J + 16 * b + i] = acc[a][b][v];
}

// Factor tile: slice t.a of the t.b slices of fact_rows rows of the factor `src` (rows x RK).
// When `dst` is set the slice is also copied there (the aggregated factor becomes the next
// step's reused factor).  A factor of one slice finishes W here; otherwise the slice's Gram is
// stored as a partial and K_CHOL adds the partials and finishes W.  From kBlockedRank on the
// Gram always goes to a partial (its blocks on and above the diagonal), K_GSUM adds and mirrors
// the partials and K_CHOL finishes W.
template <int RK>
__device__ void fact_tile(const KArgs& a, const Tile& t, const float* src, float* dst, int64_t rows) {
  const MatDesc d = a.mats[t.idx];
  if (a.copy_only) {  // Power-SGD keeps the aggregated Q as it is: copied, no W
    const int sl = RK >= kBlockedRank ? (t.a & 0xffff) : t.a;
    if (!dst || (RK >= kBlockedRank && (t.a >> 16) != 0)) return;
    const int64_t r0 = static_cast<int64_t>(sl) * d.fact_rows;
    const int64_t r1 = r0 + d.fact_rows < rows ? r0 + d.fact_rows : rows;
    for (int64_t e = r0 * RK + tid(); e < r1 * RK; e += static_cast<int64_t>(blockDim.x)) dst[e] = src[e];
    return;
  }
  if constexpr (RK >= kBlockedRank) {  // always a partial: K_CHOL forms W
    const int sl = t.a & 0xffff, part = t.a >> 16;
    const int64_t r0 = static_cast<int64_t>(sl) * d.fact_rows;
    const int64_t r1 = r0 + d.fact_rows < rows ? r0 + d.fact_rows : rows;
    gram_blocked<RK>(src, r0, r1, a.gpart + d.gpart + static_cast<int64_t>(sl) * RK * RK, dst, part);
  } else {
    const int64_t r0 = static_cast<int64_t>(t.a) * d.fact_rows;
    const int64_t r1 = r0 + d.fact_rows < rows ? r0 + d.fact_rows : rows;
    __shared__ double G[RK * RK];
    gram_rows<RK>(src, r0, r1, G, dst);
    if (t.b == 1) {
      cholesky_w<RK>(G, a.w + d.w_slot);
    } else {
      double* part = a.gpart + d.gpart + static_cast<int64_t>(t.a) * RK * RK;
      for (int e = tid(); e < RK * RK; e += kBlock) part[e] = G[e];
    }
  }
}

}  // namespace
}  // namespace acp
