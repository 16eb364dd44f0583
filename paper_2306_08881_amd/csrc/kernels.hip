// gfx950 kernels of the ACP-SGD compressor (arXiv 2306.08881, Algorithms 1 and 2).
//
// Every kernel runs 256-thread workgroups (4 waves of 64) over a table of tiles; one
// workgroup per tile.  All reductions are deterministic: fixed-order wave butterflies,
// fixed-order sums across waves and a last-arriving-workgroup reduction that adds the
// per-tile partial sums in tile order (no floating-point atomics), so that every rank of a
// data-parallel job computes bitwise the same orthogonalised factor.
//
// Error-feedback residual of a Q-step (E_t = M' - P_hat Q_t^T) is kept in deferred form:
// the Q-step writes F = M' into the E arena and the next P-step subtracts the rank-r term
// P_hat Q_loc^T while it streams F, so each step reads M and E once and writes E once.
#include <hip/hip_runtime.h>

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

__device__ inline float4 fma4(float s, const float4& v, const float4& acc) {
  return make_float4(fmaf(s, v.x, acc.x), fmaf(s, v.y, acc.y), fmaf(s, v.z, acc.z),
                     fmaf(s, v.w, acc.w));
}

template <typename T>
__device__ inline T ld_agent(const T* p) {
  return __hip_atomic_load(const_cast<T*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Arrival at a counter shared by `total` workgroups; true in the last one to arrive, after
// which every other workgroup's stores made before its own arrival are visible.
__device__ inline bool arrive_last(uint32_t* ctr, uint32_t total) {
  __shared__ uint32_t s_last;
  __threadfence();
  __syncthreads();
  if (tid() == 0) {
    const uint32_t prev = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    s_last = (prev + 1u == total) ? 1u : 0u;
  }
  __syncthreads();
  const bool last = s_last != 0u;
  if (last) __threadfence();
  return last;
}

__device__ inline void reset_counter(uint32_t* ctr) {
  if (tid() == 0) __hip_atomic_store(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Raw vectors: pack the gradient into the factor buffer (compress) or unpack the aggregated
// sum / p into the output bucket (decompress).
__device__ void vec_tile(const KArgs& a, const Tile& t, bool compress) {
  const VecDesc v = a.vecs[t.idx];
  const int64_t foff = a.parity ? v.fac_off_p : v.fac_off_q;
  for (int i = tid(); i < t.b; i += kBlock) {
    const int64_t k = static_cast<int64_t>(t.a) + i;
    if (compress)
      a.fbuf[foff + k] = a.grad[v.grad_off + k];
    else
      a.out[v.grad_off + k] = a.agg[foff + k] * a.inv_p;
  }
}

// ---------------------------------------------------------------------------------------
// Orthogonalisation, Gram/Cholesky form.  For a factor X (k x r) the Gram-Schmidt factor is
// orth(X) = X W with W = R^-1 and G = X^T X = R^T R (R upper triangular, positive diagonal):
// the same columns as Gram-Schmidt in exact arithmetic.  G is accumulated in fp64 from fp32
// products (exact) and factored in fp64.  A column j is dropped (its column of W is zero) when
// G_jj = 0 or its residual d_j = G_jj - sum_{i<j} R_ij^2 is at most tau^2 G_jj, i.e. when the
// residual norm is at most tau times the column norm.

template <int RK>
__device__ void cholesky_w(const double* G, double* R, int* drop, double* w_out) {
  for (int e = tid(); e < RK * RK; e += kBlock) R[e] = 0.0;
  __syncthreads();
  for (int j = 0; j < RK; ++j) {
    if (tid() == 0) {
      const double gjj = G[j * RK + j];
      double dj = gjj;
      for (int i = 0; i < j; ++i) dj -= R[i * RK + j] * R[i * RK + j];
      const bool keep = gjj > 0.0 && dj > kTau * kTau * gjj;
      drop[j] = keep ? 0 : 1;
      R[j * RK + j] = keep ? sqrt(dj) : 0.0;
    }
    __syncthreads();
    const int k = tid();
    if (k > j && k < RK && drop[j] == 0) {
      double s = G[j * RK + k];
      for (int i = 0; i < j; ++i) s -= R[i * RK + j] * R[i * RK + k];
      R[j * RK + k] = s / R[j * RK + j];
    }
    __syncthreads();
  }
  const int arow = tid();
  if (arow < RK) {
    double wr[RK];
#pragma unroll
    for (int j = 0; j < RK; ++j) {
      double v = 0.0;
      if (drop[j] == 0 && arow <= j) {
        v = (arow == j) ? 1.0 : 0.0;
#pragma unroll
        for (int i = 0; i < j; ++i)
          if (i >= arow) v -= R[i * RK + j] * wr[i];
        v /= R[j * RK + j];
      }
      wr[j] = v;
    }
#pragma unroll
    for (int j = 0; j < RK; ++j) w_out[arow * RK + j] = wr[j];
  }
}

// Slice `t.a` of `t.b` slices of factor rows: optionally copy them into `dst`, add their Gram
// into the partial slot, and in the last slice to arrive reduce the partials in slice order
// and factor the Gram into W.
template <int RK>
__device__ void fact_tile(const KArgs& a, const Tile& t, const float* src, float* dst, int64_t rows) {
  const MatDesc d = a.mats[t.idx];
  const int64_t r0 = static_cast<int64_t>(t.a) * d.fact_rows;
  const int64_t r1 = r0 + d.fact_rows < rows ? r0 + d.fact_rows : rows;
  if (dst)
    for (int64_t e = r0 * RK + tid(); e < r1 * RK; e += kBlock) dst[e] = src[e];
  double* part = a.gpart + d.gpart + static_cast<int64_t>(t.a) * RK * RK;
  if constexpr (RK <= 8) {
    constexpr int NT = RK * (RK + 1) / 2;
    double g[NT];
#pragma unroll
    for (int e = 0; e < NT; ++e) g[e] = 0.0;
    for (int64_t row = r0 + tid(); row < r1; row += kBlock) {
      double x[RK];
#pragma unroll
      for (int k = 0; k < RK; ++k) x[k] = static_cast<double>(src[row * RK + k]);
      int e = 0;
#pragma unroll
      for (int i = 0; i < RK; ++i)
#pragma unroll
        for (int j = i; j < RK; ++j, ++e) g[e] = fma(x[i], x[j], g[e]);
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
      part[i * RK + j] = s;
      part[j * RK + i] = s;
    }
  } else {
    constexpr int CH = 64;
    __shared__ float xs[CH * RK];
    double acc[(RK * RK + kBlock - 1) / kBlock];
#pragma unroll
    for (int q = 0; q < (RK * RK + kBlock - 1) / kBlock; ++q) acc[q] = 0.0;
    for (int64_t c0 = r0; c0 < r1; c0 += CH) {
      const int64_t cn = (r1 - c0) < CH ? (r1 - c0) : CH;
      for (int e = tid(); e < cn * RK; e += kBlock) xs[e] = src[c0 * RK + e];
      __syncthreads();
#pragma unroll
      for (int q = 0; q < (RK * RK + kBlock - 1) / kBlock; ++q) {
        const int e = tid() + q * kBlock;
        if (e < RK * RK) {
          const int i = e / RK, j = e % RK;
          double s = acc[q];
          for (int rr = 0; rr < cn; ++rr)
            s = fma(static_cast<double>(xs[rr * RK + i]), static_cast<double>(xs[rr * RK + j]), s);
          acc[q] = s;
        }
      }
      __syncthreads();
    }
#pragma unroll
    for (int q = 0; q < (RK * RK + kBlock - 1) / kBlock; ++q) {
      const int e = tid() + q * kBlock;
      if (e < RK * RK) part[e] = acc[q];
    }
  }
  if (!arrive_last(a.ctr + d.ctr_gram, static_cast<uint32_t>(t.b))) return;
  __shared__ double G[RK * RK];
  __shared__ double R[RK * RK];
  __shared__ int drop[RK];
  const double* gp = a.gpart + d.gpart;
  for (int e = tid(); e < RK * RK; e += kBlock) {
    double s = 0.0;
    for (int sl = 0; sl < t.b; ++sl) s += ld_agent(gp + static_cast<int64_t>(sl) * RK * RK + e);
    G[e] = s;
  }
  __syncthreads();
  cholesky_w<RK>(G, R, drop, a.w + d.w_slot);
  reset_counter(a.ctr + d.ctr_gram);
}

// Xh = X W for rows [t.a, t.a + t.b) of the P (variant 0) or Q (variant 1) slot.
template <int RK>
__global__ __launch_bounds__(kBlock) void k_apply(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  const MatDesc d = a.mats[t.idx];
  __shared__ double W[RK * RK];
  for (int e = tid(); e < RK * RK; e += kBlock) W[e] = a.w[d.w_slot + e];
  __syncthreads();
  const int64_t row = static_cast<int64_t>(t.a) + tid();
  if (tid() >= t.b) return;
  const bool q = a.variant == 1;
  const float* X = a.fac + (q ? d.q_slot : d.p_slot) + row * RK;
  float* Y = a.fac + (q ? d.qh_slot : d.ph_slot) + row * RK;
  double x[RK];
#pragma unroll
  for (int l = 0; l < RK; ++l) x[l] = static_cast<double>(X[l]);
#pragma unroll
  for (int k = 0; k < RK; ++k) {
    double s = 0.0;
#pragma unroll
    for (int l = 0; l <= k; ++l) s = fma(x[l], W[l * RK + k], s);
    Y[k] = static_cast<float>(s);
  }
}

template <int RK>
__global__ __launch_bounds__(kBlock) void k_gram(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  const MatDesc d = a.mats[t.idx];
  const bool q = a.variant == 1;
  fact_tile<RK>(a, t, a.fac + (q ? d.q_slot : d.p_slot), nullptr, q ? d.m : d.n);
}

// ---------------------------------------------------------------------------------------
// P-step, fused single pass (r = 4, rows of up to 5120 columns, 16-byte aligned rows).
// A row is split over `wpr` waves (1, 2, 3 or 4); each lane owns S float4 column groups of
// its wave's segment and keeps their rows of Qh (and of Q_loc when E is deferred) in
// registers for the whole tile.  Per row: M' = M + E (or M + F - Ph_row Q_loc^T), P = M' Qh
// reduced over the row, E = M' - P Qh^T written back, P written to the factor buffer.
template <int S>
__global__ __launch_bounds__(kBlock) void k_pfused(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  if (t.kind == T_VEC) {
    vec_tile(a, t, true);
    return;
  }
  const MatDesc d = a.mats[t.idx];
  const int m4 = d.m >> 2;
  const int wpr = d.wpr, rpr = 4 / wpr;
  const int wave = tid() >> 6, lane = tid() & 63;
  const int rsub = wave / wpr, seg = wave - rsub * wpr;
  const bool wave_on = rsub < rpr;
  const bool ef = a.ef != 0, deferred = a.deferred != 0;

  int c4[S];
  bool ok[S];
#pragma unroll
  for (int s = 0; s < S; ++s) {
    c4[s] = seg * 64 * S + s * 64 + lane;
    ok[s] = wave_on && c4[s] < m4;
  }
  const float4* Qh4 = reinterpret_cast<const float4*>(a.fac + d.qh_slot);
  const float4* Ql4 = reinterpret_cast<const float4*>(a.fac + d.ql_slot);
  float4 qh[S][4], ql[S][4];
#pragma unroll
  for (int s = 0; s < S; ++s)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      qh[s][c] = ok[s] ? Qh4[4 * c4[s] + c] : make_float4(0.f, 0.f, 0.f, 0.f);
      ql[s][c] = (ok[s] && deferred) ? Ql4[4 * c4[s] + c] : make_float4(0.f, 0.f, 0.f, 0.f);
    }

  const float4* G4 = reinterpret_cast<const float4*>(a.grad + d.grad_off);
  float4* E4 = reinterpret_cast<float4*>(a.e + d.e_off);
  const float* Ph = a.fac + d.ph_slot;
  __shared__ float4 red[4];

  const int row_end = t.a + t.b;
  for (int r0 = t.a; r0 < row_end; r0 += rpr) {
    const int row = r0 + rsub;
    const bool act = wave_on && row < row_end;
    const int64_t base = static_cast<int64_t>(row) * m4;
    float4 mp[S];
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    if (act) {
      float4 ph = make_float4(0.f, 0.f, 0.f, 0.f);
      if (deferred) ph = *reinterpret_cast<const float4*>(Ph + static_cast<int64_t>(row) * 4);
#pragma unroll
      for (int s = 0; s < S; ++s) {
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (ok[s]) {
          v = G4[base + c4[s]];
          if (ef) {
            const float4 e = E4[base + c4[s]];
            v = v + e;
          }
          if (deferred) {
            v.x -= dot4(ph, ql[s][0]);
            v.y -= dot4(ph, ql[s][1]);
            v.z -= dot4(ph, ql[s][2]);
            v.w -= dot4(ph, ql[s][3]);
          }
        }
        mp[s] = v;
        acc = fma4(v.x, qh[s][0], acc);
        acc = fma4(v.y, qh[s][1], acc);
        acc = fma4(v.z, qh[s][2], acc);
        acc = fma4(v.w, qh[s][3], acc);
      }
    }
    acc = wave_sum(acc);
    float4 P = acc;
    if (wpr > 1) {
      if (lane == 0) red[wave] = acc;
      __syncthreads();
      if (wave_on) {
        P = red[rsub * wpr];
        for (int k = 1; k < wpr; ++k) P = P + red[rsub * wpr + k];
      }
      __syncthreads();
    }
    if (act) {
      if (ef) {
#pragma unroll
        for (int s = 0; s < S; ++s)
          if (ok[s]) {
            float4 e = mp[s];
            e.x -= dot4(P, qh[s][0]);
            e.y -= dot4(P, qh[s][1]);
            e.z -= dot4(P, qh[s][2]);
            e.w -= dot4(P, qh[s][3]);
            E4[base + c4[s]] = e;
          }
      }
      if (seg == 0 && lane == 0) {
        float* dst = a.fbuf + d.fac_off_p + static_cast<int64_t>(row) * 4;
        dst[0] = P.x;
        dst[1] = P.y;
        dst[2] = P.z;
        dst[3] = P.w;
      }
    }
  }
}

// P-step, general: one workgroup per row computes P_row = M'_row Qh.
template <int RK>
__global__ __launch_bounds__(kBlock) void k_prow(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  if (t.kind == T_VEC) {
    vec_tile(a, t, true);
    return;
  }
  const MatDesc d = a.mats[t.idx];
  const int64_t row = t.a;
  const int64_t m = d.m;
  const float* G = a.grad + d.grad_off + row * m;
  const float* E = a.e + d.e_off + row * m;
  const float* Qh = a.fac + d.qh_slot;
  const float* Ql = a.fac + d.ql_slot;
  const bool ef = a.ef != 0, deferred = a.deferred != 0;
  float ph[RK];
#pragma unroll
  for (int k = 0; k < RK; ++k) ph[k] = deferred ? a.fac[d.ph_slot + row * RK + k] : 0.f;
  float acc[RK];
#pragma unroll
  for (int k = 0; k < RK; ++k) acc[k] = 0.f;
  for (int64_t j = tid(); j < m; j += kBlock) {
    float mp = G[j];
    if (ef) mp += E[j];
    if (deferred)
#pragma unroll
      for (int k = 0; k < RK; ++k) mp -= ph[k] * Ql[j * RK + k];
#pragma unroll
    for (int k = 0; k < RK; ++k) acc[k] = fmaf(mp, Qh[j * RK + k], acc[k]);
  }
  __shared__ float red[4][RK];
#pragma unroll
  for (int k = 0; k < RK; ++k) acc[k] = wave_sum(acc[k]);
  if ((tid() & 63) == 0)
#pragma unroll
    for (int k = 0; k < RK; ++k) red[tid() >> 6][k] = acc[k];
  __syncthreads();
  if (tid() < RK) {
    const int k = tid();
    a.fbuf[d.fac_off_p + row * RK + k] = ((red[0][k] + red[1][k]) + red[2][k]) + red[3][k];
  }
}

// P-step, general: E = M' - P Qh^T over a tile of rows (P from the factor buffer).
template <int RK>
__global__ __launch_bounds__(kBlock) void k_eupd(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  const MatDesc d = a.mats[t.idx];
  const int64_t m = d.m;
  const bool deferred = a.deferred != 0;
  const float* Qh = a.fac + d.qh_slot;
  const float* Ql = a.fac + d.ql_slot;
  const float* Ph = a.fac + d.ph_slot;
  const float* P = a.fbuf + d.fac_off_p;
  const int64_t total = static_cast<int64_t>(t.b) * m;
  for (int64_t e = tid(); e < total; e += kBlock) {
    const int64_t row = t.a + e / m, j = e % m;
    const int64_t idx = row * m + j;
    float mp = a.grad[d.grad_off + idx] + a.e[d.e_off + idx];
    if (deferred)
#pragma unroll
      for (int k = 0; k < RK; ++k) mp -= Ph[row * RK + k] * Ql[j * RK + k];
    float r = mp;
#pragma unroll
    for (int k = 0; k < RK; ++k) r -= P[row * RK + k] * Qh[j * RK + k];
    a.e[d.e_off + idx] = r;
  }
}

// Write E (explicit, or F - Ph Q_loc^T when deferred) of a tile of rows into a bucket-shaped
// output.
template <int RK>
__global__ __launch_bounds__(kBlock) void k_emat(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  const MatDesc d = a.mats[t.idx];
  const int64_t m = d.m;
  const bool deferred = a.deferred != 0;
  const float* Ql = a.fac + d.ql_slot;
  const float* Ph = a.fac + d.ph_slot;
  const int64_t total = static_cast<int64_t>(t.b) * m;
  for (int64_t e = tid(); e < total; e += kBlock) {
    const int64_t row = t.a + e / m, j = e % m;
    const int64_t idx = row * m + j;
    float v = a.e[d.e_off + idx];
    if (deferred)
#pragma unroll
      for (int k = 0; k < RK; ++k) v -= Ph[row * RK + k] * Ql[j * RK + k];
    a.out[d.grad_off + idx] = v;
  }
}

// ---------------------------------------------------------------------------------------
// Q-step: tile = (row chunk, column block).  Each lane owns CPT adjacent columns; the four
// waves take every fourth row of the chunk.  F = M' is written back (deferred E) and the
// partial M'^T Ph of the tile is summed across waves in wave order; the last row chunk to
// arrive for a column block adds the chunks' partials in chunk order, giving Q_loc, which is
// written to the factor buffer and to the Ql slot.
template <int RK, int CPT>
__global__ __launch_bounds__(kBlock) void k_qstep(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  if (t.kind == T_VEC) {
    vec_tile(a, t, true);
    return;
  }
  const MatDesc d = a.mats[t.idx];
  const int wave = tid() >> 6, lane = tid() & 63;
  const int64_t m = d.m;
  const int64_t r0 = static_cast<int64_t>(t.a) * d.q_rows;
  const int64_t r1 = (r0 + d.q_rows < d.n) ? r0 + d.q_rows : d.n;
  const int64_t col = static_cast<int64_t>(t.b) * d.q_cb + lane * CPT;
  const bool valid = col < m;
  const bool ef = a.ef != 0;
  const float* G = a.grad + d.grad_off;
  float* E = a.e + d.e_off;
  const float* Ph = a.fac + d.ph_slot;
  float acc[CPT][RK];
#pragma unroll
  for (int c = 0; c < CPT; ++c)
#pragma unroll
    for (int k = 0; k < RK; ++k) acc[c][k] = 0.f;
  for (int64_t row = r0 + wave; row < r1; row += 4) {
    float ph[RK];
#pragma unroll
    for (int k = 0; k < RK; ++k) ph[k] = Ph[row * RK + k];
    if (valid) {
      float mp[CPT];
      const int64_t idx = row * m + col;
      if constexpr (CPT == 4) {
        float4 g = *reinterpret_cast<const float4*>(G + idx);
        if (ef) {
          const float4 e = *reinterpret_cast<const float4*>(E + idx);
          g = g + e;
          *reinterpret_cast<float4*>(E + idx) = g;
        }
        mp[0] = g.x;
        mp[1] = g.y;
        mp[2] = g.z;
        mp[3] = g.w;
      } else {
        float g = G[idx];
        if (ef) {
          g += E[idx];
          E[idx] = g;
        }
        mp[0] = g;
      }
#pragma unroll
      for (int c = 0; c < CPT; ++c)
#pragma unroll
        for (int k = 0; k < RK; ++k) acc[c][k] = fmaf(mp[c], ph[k], acc[c][k]);
    }
  }
  constexpr int W = 64 * CPT * RK;  // partial entries of one wave
  __shared__ float red[4][W];
#pragma unroll
  for (int c = 0; c < CPT; ++c)
#pragma unroll
    for (int k = 0; k < RK; ++k) red[wave][(lane * CPT + c) * RK + k] = acc[c][k];
  __syncthreads();
  const int64_t ncb = (m + d.q_cb - 1) / d.q_cb;
  const int64_t stride = ncb * d.q_cb * RK;  // one row chunk of partials
  float* part = a.qpart + d.qpart + static_cast<int64_t>(t.a) * stride + static_cast<int64_t>(t.b) * d.q_cb * RK;
  for (int e = tid(); e < W; e += kBlock) part[e] = ((red[0][e] + red[1][e]) + red[2][e]) + red[3][e];
  if (!arrive_last(a.ctr + d.ctr_q + t.b, static_cast<uint32_t>(d.q_chunks))) return;
  const float* base = a.qpart + d.qpart + static_cast<int64_t>(t.b) * d.q_cb * RK;
  for (int e = tid(); e < W; e += kBlock) {
    const int64_t c = static_cast<int64_t>(t.b) * d.q_cb + e / RK;
    if (c >= m) continue;
    float s = 0.f;
    for (int ch = 0; ch < d.q_chunks; ++ch) s += ld_agent(base + ch * stride + e);
    const int64_t o = c * RK + (e % RK);
    a.fbuf[d.fac_off_q + o] = s;
    a.fac[d.ql_slot + o] = s;
  }
  reset_counter(a.ctr + d.ctr_q + t.b);
}

// ---------------------------------------------------------------------------------------
// Decompress: M_hat = A B^T / p over a tile of rows.  Odd step: A = P_agg (factor buffer),
// B = Qh; even step: A = Ph, B = Q_agg.  B is staged in LDS column-major in chunks.  Factor
// tiles keep the aggregated factor as the next step's reused factor and build its W.
template <int RK, int VW>
__global__ __launch_bounds__(kBlock) void k_recon(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  const bool odd = a.parity != 0;
  if (t.kind == T_VEC) {
    vec_tile(a, t, false);
    return;
  }
  const MatDesc d = a.mats[t.idx];
  if (t.kind == T_FACT) {
    const float* src = a.agg + (odd ? d.fac_off_p : d.fac_off_q);
    float* dst = a.fac + (odd ? d.p_slot : d.q_slot);
    fact_tile<RK>(a, t, src, dst, odd ? d.n : d.m);
    return;
  }
  constexpr int CK = (8192 / RK) < 4096 ? (8192 / RK) : 4096;
  __shared__ __align__(16) float Bs[RK * CK];
  const float* A = odd ? a.agg + d.fac_off_p : a.fac + d.ph_slot;
  const float* B = odd ? a.fac + d.qh_slot : a.agg + d.fac_off_q;
  const int wave = tid() >> 6, lane = tid() & 63;
  const int64_t m = d.m;
  float* O = a.out + d.grad_off;
  for (int64_t c0 = 0; c0 < m; c0 += CK) {
    const int cw = static_cast<int>((m - c0) < CK ? (m - c0) : CK);
    for (int e = tid(); e < cw * RK; e += kBlock) {
      const int j = e / RK, k = e - j * RK;
      Bs[k * CK + j] = B[(c0 + j) * RK + k];
    }
    __syncthreads();
    for (int64_t row = t.a + wave; row < t.a + t.b; row += 4) {
      float ar[RK];
#pragma unroll
      for (int k = 0; k < RK; ++k) ar[k] = A[row * RK + k] * a.inv_p;
      if constexpr (VW == 4) {
        for (int j4 = lane; j4 < (cw >> 2); j4 += 64) {
          float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
          for (int k = 0; k < RK; ++k)
            o = fma4(ar[k], *reinterpret_cast<const float4*>(&Bs[k * CK + 4 * j4]), o);
          *reinterpret_cast<float4*>(O + row * m + c0 + 4 * j4) = o;
        }
      } else {
        for (int j = lane; j < cw; j += 64) {
          float o = 0.f;
#pragma unroll
          for (int k = 0; k < RK; ++k) o = fmaf(ar[k], Bs[k * CK + j], o);
          O[row * m + c0 + j] = o;
        }
      }
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(kBlock) void k_vec(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  vec_tile(a, t, true);
}

template <int RK>
hipError_t launch_rank(const Launch& l, const KArgs& args, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(l.ntiles)), block(kBlock);
  switch (l.kernel) {
    case K_APPLY: hipLaunchKernelGGL(k_apply<RK>, grid, block, 0, s, args); break;
    case K_PROW: hipLaunchKernelGGL(k_prow<RK>, grid, block, 0, s, args); break;
    case K_EUPD: hipLaunchKernelGGL(k_eupd<RK>, grid, block, 0, s, args); break;
    case K_EMAT: hipLaunchKernelGGL(k_emat<RK>, grid, block, 0, s, args); break;
    case K_GRAM: hipLaunchKernelGGL(k_gram<RK>, grid, block, 0, s, args); break;
    case K_QSTEP:
      if (l.variant == 4) {
        if constexpr (RK <= 8) {
          hipLaunchKernelGGL((k_qstep<RK, 4>), grid, block, 0, s, args);
        } else {
          return hipErrorInvalidValue;
        }
      } else {
        hipLaunchKernelGGL((k_qstep<RK, 1>), grid, block, 0, s, args);
      }
      break;
    case K_RECON:
      if (l.variant == 4)
        hipLaunchKernelGGL((k_recon<RK, 4>), grid, block, 0, s, args);
      else
        hipLaunchKernelGGL((k_recon<RK, 1>), grid, block, 0, s, args);
      break;
    case K_PFUSED:
      if constexpr (RK == 4) {
        switch (l.variant) {
          case 1: hipLaunchKernelGGL(k_pfused<1>, grid, block, 0, s, args); break;
          case 2: hipLaunchKernelGGL(k_pfused<2>, grid, block, 0, s, args); break;
          case 3: hipLaunchKernelGGL(k_pfused<3>, grid, block, 0, s, args); break;
          case 4: hipLaunchKernelGGL(k_pfused<4>, grid, block, 0, s, args); break;
          case 5: hipLaunchKernelGGL(k_pfused<5>, grid, block, 0, s, args); break;
          default: return hipErrorInvalidValue;
        }
        break;
      } else {
        return hipErrorInvalidValue;
      }
    case K_VEC: hipLaunchKernelGGL(k_vec, grid, block, 0, s, args); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch(const Launch& l, int32_t rank, const KArgs& args, hipStream_t s) {
  if (l.ntiles <= 0) return hipSuccess;
  switch (rank) {
    case 1: return launch_rank<1>(l, args, s);
    case 2: return launch_rank<2>(l, args, s);
    case 4: return launch_rank<4>(l, args, s);
    case 8: return launch_rank<8>(l, args, s);
    case 16: return launch_rank<16>(l, args, s);
    case 32: return launch_rank<32>(l, args, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace acp
