// gfx950 kernels of the ACP-SGD compressor (arXiv 2306.08881, Algorithms 1 and 2): the
// rank-4 register-resident streaming kernels, the general kernels for ranks 1 and 2 and for
// matrices the rank-4 kernels do not take, the Q-step finish, the factor tiles and the launch
// dispatch.  The MFMA kernels of ranks 8, 16 and 32 are in wide.hip.
//
// Every kernel runs 256-thread workgroups (4 waves of 64) over a table of tiles; one
// workgroup per tile.  Workgroups never wait for each other: a reduction that spans
// workgroups writes per-tile partial sums and a later kernel of the same stream adds them in
// tile order.  Together with fixed-order wave butterflies and fixed-order sums across waves
// this makes every result bitwise reproducible, which a data-parallel job needs so that all
// ranks keep the same orthogonalised factor.
//
// The error-feedback residual of a Q-step (E_t = M' - P_hat Q_t^T) is kept in deferred form:
// the Q-step writes F = M' into the E arena and the next P-step subtracts the rank-r term
// P_hat Q_loc^T while it streams F, so each step reads M and E once and writes E once.
#include "device.hpp"

#include <mutex>
#include <vector>

namespace acp {

hipError_t launch_wide(const Launch& l, int32_t rank, const KArgs& args, hipStream_t s);

namespace {

// Factor tiles alone: W of the P (variant bit 0 clear) or Q factor of a matrix, read from its slot,
// or with kFactFromBuffer from the aggregated factor buffer and copied into the slot.
template <int RK>
__global__ __launch_bounds__(kBlock) void k_fact(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  const MatDesc d = a.mats[t.idx];
  const bool q = (a.variant & 1) != 0;
  float* slot = a.fac + (q ? d.q_slot : d.p_slot);
  if (a.variant & kFactFromBuffer)
    fact_tile<RK>(a, t, src_of(a, d.bucket) + (q ? d.fac_off_q : d.fac_off_p), slot, q ? d.m : d.n);
  else
    fact_tile<RK>(a, t, slot, nullptr, q ? d.m : d.n);
}

// No reuse (the ablation of Section V-B): the factor a step would have reused is drawn anew, i.i.d.
// standard normal, from the initial factors' counter-based generator with the step in the high
// half of the key: element i (row-major) of factor f (0: P, 1: Q) of tensor k at step t takes the
// SplitMix64 outputs x = mix(s + (2i + 1) g), y = mix(s + (2i + 2) g) of the stream
// s = mix(seed ^ mix(t 2^32 + 2k + f)) and becomes sqrt(-2 ln u1) cos(2 pi u2) in fp64 with
// u1 = ((x >> 11) + 1) 2^-53, u2 = (y >> 11) 2^-53, rounded to fp32.  Tile: factor rows
// [t.a, t.a + t.b) of the P (variant 0) or Q (variant 1) slot.
__device__ inline uint64_t splitmix_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

template <int RK>
__global__ __launch_bounds__(kBlock) void k_draw(KArgs a) {
  constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
  constexpr double kTwoPi = 2.0 * 3.14159265358979323846;
  const Tile t = a.tiles[blockIdx.x];
  const MatDesc d = a.mats[t.idx];
  const uint64_t f = static_cast<uint64_t>(a.variant & 1);
  float* slot = a.fac + (f ? d.q_slot : d.p_slot);
  const uint64_t key = (static_cast<uint64_t>(a.step) << 32) + 2ull * static_cast<uint64_t>(d.tid) + f;
  const uint64_t s = splitmix_mix(a.seed ^ splitmix_mix(key));
  const int64_t e0 = static_cast<int64_t>(t.a) * RK, ne = static_cast<int64_t>(t.b) * RK;
  for (int64_t k = tid(); k < ne; k += kBlock) {
    const uint64_t i = static_cast<uint64_t>(e0 + k);
    const uint64_t x = splitmix_mix(s + (2ull * i + 1ull) * kGamma);
    const uint64_t y = splitmix_mix(s + (2ull * i + 2ull) * kGamma);
    const double u1 = static_cast<double>((x >> 11) + 1ull) * 0x1.0p-53;
    const double u2 = static_cast<double>(y >> 11) * 0x1.0p-53;
    const double rad = sqrt(-2.0 * log(u1));
    const double ang = cos(kTwoPi * u2);
    slot[e0 + k] = static_cast<float>(rad * ang);
  }
}

// Power-SGD's first half with error feedback: the E arena receives M' = M + E_{t-1}, the image of
// the bucket that both of the step's products then read, E_{t-1} taken in the form the arena holds
// it (E itself, or F - Ph Q_loc^T after a Q-step).  T_QTILE tiles: `rows` rows from t.a and
// kImageCols columns of a matrix, one thread per column; the tile's rows of the term's row factor
// sit in LDS and, up to rank 32, the thread's column-factor row in registers.  T_VEC tiles copy
// raw vectors into their arena slots; T_FACT tiles set W = I, so that the P-step kernels multiply
// by Q_{t-1} itself.
template <int RK>
__global__ __launch_bounds__(kBlock) void k_image(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  if (t.kind == T_FACT) {
    const MatDesc d = a.mats[t.idx];
    for (int e = tid(); e < RK * RK; e += kBlock) a.w[d.w_slot + e] = (e / RK == e % RK) ? 1.0 : 0.0;
    return;
  }
  if (t.kind == T_VEC) {
    const VecDesc v = a.vecs[t.idx];
    const float* src = src_of(a, v.bucket) + v.grad_off + t.a;
    float* dst = a.e + v.e_off + t.a;
    for (int i = tid(); i < t.b; i += kBlock) dst[i] = src[i];
    return;
  }
  const MatDesc d = a.mats[t.idx];
  const int cb = t.b & 0xffff, rows = t.b >> 16;
  const int64_t m = d.m;
  const int64_t c = static_cast<int64_t>(cb) * kImageCols + tid();
  const bool fform = deferred_of(a, d.bucket), xform = deferred_p_of(a, d.bucket);
  const bool term = fform || xform;
  const float* L = a.fac + (xform ? d.qh_slot : d.ql_slot);  // column factor of the term (m x r)
  const float* R = a.fac + (xform ? d.pl_slot : d.ph_slot);  // row factor of the term (n x r)
  __shared__ float rs[4096];  // the tile's rows of R (rows * RK <= 4096)
  if (term)
    for (int e = tid(); e < rows * RK; e += kBlock) rs[e] = R[static_cast<int64_t>(t.a) * RK + e];
  __syncthreads();
  if (c >= m) return;
  constexpr int KR = RK <= 32 ? RK : 32;  // ranks of the column-factor row held in registers
  float l[KR];
#pragma unroll
  for (int k = 0; k < KR; ++k) l[k] = term ? L[c * RK + k] : 0.f;
  const float* M = src_of(a, d.bucket) + d.grad_off;
  float* X = a.e + d.e_off;
  for (int i = 0; i < rows; ++i) {
    const int64_t idx = (static_cast<int64_t>(t.a) + i) * m + c;
    float v = M[idx] + X[idx];
    if (term) {
#pragma unroll
      for (int k = 0; k < KR; ++k) v -= rs[i * RK + k] * l[k];
      for (int k = KR; k < RK; ++k) v -= rs[i * RK + k] * L[c * RK + k];
    }
    X[idx] = v;
  }
}

// Cholesky G = R^T R and W = R^-1 of a Gram matrix in shared memory (RK = 128, row-major; only
// the upper triangle is read) for ranks from kBlockedRank on, by the whole workgroup, in blocks
// of 32.  For each diagonal block K in order:
//   (i)   one wave factors the block (lane j keeps column j in registers; at pivot p every lane
//         takes the drop test, forms R[p][j] and updates its column with row p of R, which the
//         lanes pass through LDS) and forms W_KK = R_KK^-1 by rows (lane j, row j);
//   (ii)  the block row right of it: R_KJ = W_KK^T G_KJ (with dropped pivots W_KK's zero columns
//         give R's zero rows, as forward substitution over the kept pivots would);
//   (iii) the trailing upper triangle: G_IJ -= R_KI^T R_KJ.
// These are the pivots of the unblocked right-looking form, in the same order.  Then block column
// J of W (J = 1, 2, 3) from the earlier ones: W_IJ = -(sum_{I <= L < J} W_IL R_LJ) W_JJ.  W[i][c]
// (i < c) is kept in the strictly lower triangle at G[RK-1-i][RK-1-c] and its diagonal apart.
// Dropped pivots give zero rows and columns of R and W.  G[] is overwritten.  The drop test
// compares with the diagonal gref[i * gstride] (G's own unless given: a trailing block of a
// larger Gram matrix is tested against that matrix's diagonal); W goes to w_out with rows ldw
// apart.
template <int RK>
__device__ __attribute__((always_inline)) void cholesky_w_blocked(double* G, double* w_out, int ldw = RK,
                                                                const double* gref = nullptr, int gstride = 0) {
  static_assert(RK == 128 && kBlock == 256, "4 x 4 blocks of 32 on 256 threads");
  constexpr int B = 32, NBK = RK / B;
  __shared__ double g0[RK], wdiag[RK], rowb[B];
  __shared__ double T[(RK - B) * B];  // one block column's W[0:k0][.] R[.][block] products
  auto wl = [&](int i, int c) -> double& { return G[(RK - 1 - i) * RK + (RK - 1 - c)]; };  // W[i][c], i < c
  for (int i = tid(); i < RK; i += kBlock) g0[i] = gref ? gref[i * gstride] : G[i * RK + i];
  __syncthreads();
  const int lane = tid() & 63;
  for (int K = 0; K < NBK; ++K) {
    const int k0 = K * B, nc = RK - k0 - B;  // columns right of the block
    // (i) the diagonal block on the first wave
    if (tid() < B) {
      const int j = lane;
      double g[B];
#pragma unroll
      for (int a = 0; a < B; ++a) g[a] = a <= j ? G[(k0 + a) * RK + k0 + j] : 0.0;
      const double refl = g0[k0 + j];  // pivot j's reference diagonal, read by lane
#pragma unroll
      for (int p = 0; p < B; ++p) {
        asm volatile("" ::: "memory");  // one pivot at a time
        const double dk = readlane_d(g[p], p);
        const double ref = readlane_d(refl, p);
        const bool keep = ref > 0.0 && dk > kTau * kTau * ref;
        const double rkk = keep ? sqrt(dk) : 0.0, rinv = keep ? 1.0 / rkk : 0.0;
        const double rpj = j > p ? g[p] * rinv : (j == p ? rkk : 0.0);
        g[p] = rpj;  // row p of R
        if (j == 0) wdiag[k0 + p] = rinv;  // W's diagonal: 1 / R[p][p], zero when dropped
        if (keep) {
          // row p goes to every lane through LDS (one wave: its LDS accesses keep their order)
          rowb[j] = rpj;
          asm volatile("" ::: "memory");
#pragma unroll
          for (int a = p + 1; a < B; ++a) g[a] -= rowb[a] * rpj;
        }
      }
#pragma unroll
      for (int a = 0; a < B; ++a)
        if (a <= j) G[(k0 + a) * RK + k0 + j] = g[a];
      // W_KK row a = j: W[a][c] = -(sum_{l < c} W[a][l] R[l][c]) / R[c][c] for c > a (zero for
      // l < a), read back from LDS one column of R at a time
      const double* R = G + k0 * RK + k0;
      double w[B];
#pragma unroll
      for (int c = 0; c < B; ++c) {
        asm volatile("" ::: "memory");  // this column's loads only
        double s = 0.0;
#pragma unroll
        for (int l = 0; l < c; ++l) s += w[l] * R[l * RK + c];
        const double rinv = wdiag[k0 + c];
        w[c] = c < j ? 0.0 : (c == j ? rinv : -s * rinv);
      }
#pragma unroll
      for (int c = 0; c < B; ++c)
        if (c > j) wl(k0 + j, k0 + c) = w[c];
    }
    __syncthreads();
    if (nc == 0) break;
    // (ii) R_KJ = W_KK^T G_KJ: entry (k0 + a, k0 + B + c), a sum over b <= a
    {
      constexpr int QN = B * (RK - B) / kBlock;
      double res[QN];
#pragma unroll
      for (int q = 0; q < QN; ++q) {
        const int e = tid() + q * kBlock, a = e / nc, c = e % nc;
        double v = 0.0;
        if (e < B * nc) {
          const int j = k0 + B + c;
          double s2[2] = {wdiag[k0 + a] * G[(k0 + a) * RK + j], 0.0};
          for (int b = 0; b < a; ++b) s2[b & 1] += wl(k0 + b, k0 + a) * G[(k0 + b) * RK + j];
          v = s2[0] + s2[1];
        }
        res[q] = v;
      }
      __syncthreads();
#pragma unroll
      for (int q = 0; q < QN; ++q) {
        const int e = tid() + q * kBlock;
        if (e < B * nc) G[(k0 + e / nc) * RK + k0 + B + e % nc] = res[q];
      }
      __syncthreads();
    }
    // (iii) the trailing upper triangle: G[i][j] -= sum_a R[k0 + a][i] R[k0 + a][j], i <= j, on
    // the fp64 matrix cores in 16 x 16 tiles (tiles ti <= tj, tile t on wave t % 4; one
    // v_mfma_f64_16x16x4f64 per four rows a); entries below the diagonal of a diagonal tile are
    // not written (that triangle keeps W)
    {
      const int nt = nc / 16, w = tid() / kWave, li = lane % 16, lk = lane / 16, c0 = k0 + B;
      int t = 0;
      for (int ti = 0; ti < nt; ++ti)
        for (int tj = ti; tj < nt; ++tj, ++t) {
          if (t % (kBlock / kWave) != w) continue;
          v4d acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
          for (int s4 = 0; s4 < B / 4; ++s4) {
            const double* r = G + (k0 + 4 * s4 + lk) * RK + c0 + li;
            acc = __builtin_amdgcn_mfma_f64_16x16x4f64(r[16 * ti], r[16 * tj], acc, 0, 0, 0);
          }
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int i = c0 + 16 * ti + 4 * v + lk, j = c0 + 16 * tj + li;
            if (i <= j) G[i * RK + j] -= acc[v];
          }
        }
    }
    __syncthreads();
  }
  // block columns of W: T = W[0:k0][0:k0] R[0:k0][block], then W[0:k0][block] = -T W_JJ, both
  // on the fp64 matrix cores in 16 x 16 tiles (tile t of the k0 / 16 x 2 on wave t % 4; one
  // v_mfma_f64_16x16x4f64 per four ranks, the operands of W taken from its triangle: zero below
  // the diagonal, wdiag on it)
  {
    const int w = tid() / kWave, li = lane % 16, lk = lane / 16;
    auto wv = [&](int r, int c) { return c > r ? wl(r, c) : (c == r ? wdiag[r] : 0.0); };  // W[r][c]
    for (int J = 1; J < NBK; ++J) {
      const int k0 = J * B, nt = 2 * (k0 / 16);
      for (int t = w; t < nt; t += kBlock / kWave) {
        const int i0 = 16 * (t / 2), c0 = 16 * (t % 2);
        v4d acc = {0.0, 0.0, 0.0, 0.0};
        for (int l0 = i0; l0 < k0; l0 += 4)  // W[i][l] is zero for l < i
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64(wv(i0 + li, l0 + lk), G[(l0 + lk) * RK + k0 + c0 + li],
                                                     acc, 0, 0, 0);
#pragma unroll
        for (int v = 0; v < 4; ++v) T[(i0 + 4 * v + lk) * B + c0 + li] = acc[v];
      }
      __syncthreads();
      for (int t = w; t < nt; t += kBlock / kWave) {
        const int i0 = 16 * (t / 2), c0 = 16 * (t % 2);
        v4d acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
        for (int q0 = 0; q0 < B; q0 += 4)
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64(T[(i0 + li) * B + q0 + lk], wv(k0 + q0 + lk, k0 + c0 + li),
                                                     acc, 0, 0, 0);
#pragma unroll
        for (int v = 0; v < 4; ++v) wl(i0 + 4 * v + lk, k0 + c0 + li) = -acc[v];
      }
      __syncthreads();
    }
  }
  for (int e = tid(); e < RK * RK; e += kBlock) {
    const int i = e / RK, c = e % RK;
    w_out[i * ldw + c] = i < c ? wl(i, c) : (i == c ? wdiag[c] : 0.0);
  }
}

// C = C0 + sg A B for 128 x 128 fp64 blocks in global or shared memory (sg = +1 or -1; C0 = 0
// when c0 is null, else C0[i][j] = c0[i * ldc + j]), by the whole workgroup on the fp64 matrix
// cores: wave w forms the 64 x 64 quadrant at rows 64 (w / 2), columns 64 (w % 2) as 4 x 4
// products of 16 x 16 (v_mfma_f64_16x16x4f64; operand entry [i][k] on lane i + 16 k, result
// entry [4 v + l / 16][l % 16] in item v of lane l), each entry C0 plus a sum over k < 128 in
// increasing groups of four, with A[i][k] = A[i * ai + k * ak] and B[k][j] = B[k * bk + j];
// store(i, j, value) takes the entries.  The next group's operands are requested before the
// current group's products.
template <typename Store>
__device__ void mm128(const double* A, int ai, int ak, const double* B, int bk, const double* c0, int ldc,
                      double sg, Store store) {
  static_assert(kBlock == 4 * kWave, "one 64 x 64 quadrant per wave");
  const int lane = tid() % kWave, i = lane % 16, k = lane / 16;
  const int i0 = 64 * (tid() / kWave / 2), j0 = 64 * (tid() / kWave % 2);
  v4d acc[4][4];
#pragma unroll
  for (int ra = 0; ra < 4; ++ra)
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        acc[ra][cb][v] = c0 ? c0[(i0 + 16 * ra + 4 * v + k) * ldc + j0 + 16 * cb + i] : 0.0;
  struct Ops {
    double a[4], b[4];
  };
  auto fetch = [&](int k0, Ops& o) {
#pragma unroll
    for (int ra = 0; ra < 4; ++ra) o.a[ra] = A[(i0 + 16 * ra + i) * ai + (k0 + k) * ak];
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) o.b[cb] = B[(k0 + k) * bk + j0 + 16 * cb + i];
  };
  auto step = [&](const Ops& o) {
#pragma unroll
    for (int ra = 0; ra < 4; ++ra)
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
        acc[ra][cb] = __builtin_amdgcn_mfma_f64_16x16x4f64(sg * o.a[ra], o.b[cb], acc[ra][cb], 0, 0, 0);
  };
  // 32 groups of four, taken in pairs; past the last pair the request repeats the last group
  Ops o0, o1;
  fetch(0, o0);
  for (int k0 = 0; k0 < 128; k0 += 8) {
    fetch(k0 + 4, o1);
    __builtin_amdgcn_sched_barrier(0);  // requests ahead of the products that do not need them
    step(o0);
    __builtin_amdgcn_sched_barrier(0);
    fetch(k0 + 8 < 128 ? k0 + 8 : 124, o0);
    __builtin_amdgcn_sched_barrier(0);
    step(o1);
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int ra = 0; ra < 4; ++ra)
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int v = 0; v < 4; ++v) store(i0 + 16 * ra + 4 * v + k, j0 + 16 * cb + i, acc[ra][cb][v]);
}

// Dst[e] = Src[(e / C) * lds + e % C] for e < R * C (R x C doubles from global memory into shared
// memory), by the whole workgroup; each thread requests 16 entries before it stores them (one
// request in flight at a time costs a memory latency per entry).
template <int R, int C>
__device__ void rows_to_lds(double* Dst, const double* Src, int lds) {
  constexpr int PT = R * C / kBlock, U = 16;
  static_assert(PT % U == 0, "whole batches");
#pragma unroll 1
  for (int c = 0; c < PT; c += U) {
    double v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = tid() + (c + u) * kBlock;
      v[u] = Src[(e / C) * lds + e % C];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) Dst[tid() + (c + u) * kBlock] = v[u];
  }
}

// W = R^-1 of a 256 x 256 Gram matrix G (global memory: the matrix's first Gram partial, which
// holds the slices' sum) in 2 x 2 blocks of 128, from the factorisation
//   G11 = R11^T R11,  R12 = R11^-T G12,  G22 - R12^T R12 = R22^T R22,
//   W11 = R11^-1,  W22 = R22^-1,  W12 = -W11 R12 W22,  W21 = 0,
// the same pivots in the same order as the unblocked form.  With dropped pivots R11^-T G12 is
// W11^T G12 (W11's zero columns give R12's zero rows) and the pivots of the second block are
// tested against G's own diagonal.  R12 (called Y) is kept in G's lower left block, which the
// upper triangle makes redundant; the shared block S holds G11, then G22 - Y^T Y, then Y W22.
__device__ void chol_split(double* G, double* W, double* S) {
  constexpr int N = 256, H = 128;
  rows_to_lds<H, H>(S, G, N);
  __syncthreads();
  cholesky_w_blocked<H>(S, W, N);  // W11
  __syncthreads();
  double* Y = G + H * N;  // Y[i][j] at Y[i * N + j]
  // Y = W11^T G12
  mm128(W, 1, N, G + H, N, nullptr, 0, 1.0, [&](int i, int j, double v) { Y[i * N + j] = v; });
  __syncthreads();
  // S = G22 - Y^T Y
  mm128(Y, 1, N, Y, N, G + H * N + H, N, -1.0, [&](int i, int j, double v) { S[i * H + j] = v; });
  __syncthreads();
  cholesky_w_blocked<H>(S, W + H * N + H, N, G + H * N + H, N + 1);  // W22
  __syncthreads();
  // S = Y W22
  mm128(Y, N, 1, W + H * N + H, N, nullptr, 0, 1.0, [&](int i, int j, double v) { S[i * H + j] = v; });
  __syncthreads();
  // W12 = -W11 (Y W22)
  mm128(W, N, 1, S, H, nullptr, 0, -1.0, [&](int i, int j, double v) { W[i * N + H + j] = v; });
  for (int e = tid(); e < H * H; e += kBlock) W[(H + e / H) * N + e % H] = 0.0;
}

// From kBlockedRank on: entries [t.a kGsumEntries, ...) of a matrix's Gram, the sum of its t.b
// slices' partials in slice order, into the first partial.  The partials hold the 4 x 4 blocks
// on and above the diagonal; the thread of an entry of a block above the diagonal also writes
// its mirror, so every entry is read and written by one thread only.
template <int RK>
__global__ __launch_bounds__(kBlock) void k_gsum(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  const MatDesc d = a.mats[t.idx];
  double* gp = a.gpart + d.gpart;
  constexpr int EPT = kGsumEntries / kBlock;  // entries per thread, 256 apart
  static_assert(kGsumEntries % kBlock == 0 && (RK * RK) % kGsumEntries == 0, "whole tiles");
  int64_t e[EPT];
  bool up[EPT];
  double s[EPT];
#pragma unroll
  for (int k = 0; k < EPT; ++k) {
    e[k] = static_cast<int64_t>(t.a) * kGsumEntries + tid() + k * kBlock;
    up[k] = (e[k] / RK) / 4 <= (e[k] % RK) / 4;
    s[k] = 0.0;
  }
  for (int sl = 0; sl < t.b; ++sl) {
    double v[EPT];
#pragma unroll
    for (int k = 0; k < EPT; ++k) v[k] = up[k] ? gp[static_cast<int64_t>(sl) * RK * RK + e[k]] : 0.0;
#pragma unroll
    for (int k = 0; k < EPT; ++k) s[k] += v[k];
  }
#pragma unroll
  for (int k = 0; k < EPT; ++k) {
    if (!up[k]) continue;
    const int i = static_cast<int>(e[k] / RK), j = static_cast<int>(e[k] % RK);
    gp[e[k]] = s[k];
    if (i / 4 < j / 4) gp[j * RK + i] = s[k];
  }
}

// W from the Gram partials of a matrix's t.b slices, added in slice order (from kBlockedRank on
// K_GSUM has added them into the first).
template <int RK>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(RK <= 32 ? 4 : 1))) void k_chol(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  const MatDesc d = a.mats[t.idx];
  constexpr bool SPLIT = RK >= kCholBlockRank;
  __shared__ double Gs[SPLIT ? 128 * 128 : RK * RK];
  double* gp = a.gpart + d.gpart;
  if constexpr (RK >= kBlockedRank) {
    if constexpr (SPLIT) {
      static_assert(RK == 256, "2 x 2 blocks of 128");
      chol_split(gp, a.w + d.w_slot, Gs);
    } else {
      rows_to_lds<RK, RK>(Gs, gp, RK);
      __syncthreads();
      cholesky_w_blocked<RK>(Gs, a.w + d.w_slot);
    }
  } else {
    // each entry added in slice order; per round, eight slices of all the thread's entries are
    // requested together (one round trip per eight slices)
    constexpr int EPT = (RK * RK + kBlock - 1) / kBlock;  // entries per thread
    double acc[EPT];
#pragma unroll
    for (int q = 0; q < EPT; ++q) acc[q] = 0.0;
    for (int sl = 0; sl < t.b; sl += 8) {
      double v[EPT][8];
#pragma unroll
      for (int q = 0; q < EPT; ++q) {
        const int e = tid() + q * kBlock;
#pragma unroll
        for (int w = 0; w < 8; ++w)
          v[q][w] = (e < RK * RK && sl + w < t.b) ? gp[static_cast<int64_t>(sl + w) * RK * RK + e] : 0.0;
      }
#pragma unroll
      for (int q = 0; q < EPT; ++q)
#pragma unroll
        for (int w = 0; w < 8; ++w)
          if (sl + w < t.b) acc[q] += v[q][w];
    }
#pragma unroll
    for (int q = 0; q < EPT; ++q)
      if (tid() + q * kBlock < RK * RK) Gs[tid() + q * kBlock] = acc[q];
    __syncthreads();
    cholesky_w<RK>(Gs, a.w + d.w_slot);
  }
}

// Xh = X W from kApplyMfmaRank on, for rows [t.a, t.a + rows) and the BW = min(r, 64) columns
// c0 = BW cb ... of Xh (t.b = rows | cb << 16), on the fp64 matrix cores: wave w forms rows
// 64 w ... + 63 as 4 x BW / 16 products of 16 x 16 (v_mfma_f64_16x16x4f64; operand entry
// [i][k] on lane i + 16 k, result entry [4 v + l / 16][l % 16] in item v of lane l), over the
// ranks 0 ... c0 + BW - 1 in steps of 16.  W is upper triangular: later ranks add zero, and so do the ranks from c0 + 16 (b + 1) on
// for the columns c0 + 16 b ... + 15, whose products are skipped.  Within a step, lane i + 16 k
// holds the four ranks 4 k ... + 3 of its row as one 16-byte word, and product s of the step
// takes rank 4 k + s from lane i + 16 k in both operands, so every rank enters once.  The next
// step's rows of X are requested before the current step's products.
template <int RK>
__device__ void apply_mfma(const KArgs& a, const Tile& t, const MatDesc& d) {
  constexpr int CB = RK >= 64 ? 4 : RK / 16;  // 16-column groups of the block
  static_assert(CB % 2 == 0, "the 16-rank steps are taken in pairs");
  const int rows = t.b & 0xffff, c0 = 16 * CB * (t.b >> 16);
  const int lane = tid() % kWave, i = lane % 16, k = lane / 16;
  const int rb = 64 * (tid() / kWave);
  if (rb >= rows) return;
  const bool q = a.variant == 1;
  const float* X = a.fac + (q ? d.q_slot : d.p_slot);
  float* Y = a.fac + (q ? d.qh_slot : d.ph_slot);
  const double* W = a.w + d.w_slot;
  // rows past the tile read its last row (no branch around the loads); they are not stored
  const float* xr[4];
#pragma unroll
  for (int ra = 0; ra < 4; ++ra) {
    const int r = rb + 16 * ra + i;
    xr[ra] = X + (static_cast<int64_t>(t.a) + (r < rows ? r : rows - 1)) * RK + 4 * k;
  }
  const double* wr = W + static_cast<int64_t>(4 * k) * RK + c0 + i;
  v4d acc[4][CB];
#pragma unroll
  for (int ra = 0; ra < 4; ++ra)
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) acc[ra][cb] = v4d{0.0, 0.0, 0.0, 0.0};
  // per step the W rows (from L2, where every tile of the matrix reads them) are requested
  // first, then the next step's X rows (from HBM), so that the wait for the former leaves the
  // latter in flight
  typedef float4 XBuf[4];
  auto fetch_x = [&](int k0, XBuf& b) {
#pragma unroll
    for (int ra = 0; ra < 4; ++ra) b[ra] = *reinterpret_cast<const float4*>(xr[ra] + k0);
  };
  auto step = [&](int k0, XBuf& b, int k1, XBuf& nb) {
    // column group cb of the block takes ranks up to c0 + 16 cb + 15 only (W is upper triangular)
    const int kz = k0 - c0;
    double w[4][CB];  // [s][cb]
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) w[s][cb] = wr[static_cast<int64_t>(k0 + s) * RK + 16 * cb];
    __builtin_amdgcn_sched_barrier(0);  // in this order
    fetch_x(k1, nb);
    __builtin_amdgcn_sched_barrier(0);
    // the conversions stay behind those requests
#pragma unroll
    for (int ra = 0; ra < 4; ++ra)
      asm volatile("" : "+v"(b[ra].x), "+v"(b[ra].y), "+v"(b[ra].z), "+v"(b[ra].w));
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      double xa[4];
#pragma unroll
      for (int ra = 0; ra < 4; ++ra) {
        const float4 v = b[ra];
        xa[ra] = static_cast<double>(s == 0 ? v.x : s == 1 ? v.y : s == 2 ? v.z : v.w);
      }
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        if (kz <= 16 * cb)
#pragma unroll
          for (int ra = 0; ra < 4; ++ra)
            acc[ra][cb] = __builtin_amdgcn_mfma_f64_16x16x4f64(xa[ra], w[s][cb], acc[ra][cb], 0, 0, 0);
    }
  };
  // c0 + BW ranks: an even number of 16-rank steps, taken in pairs; past the last pair the X
  // request repeats the last step's ranks, unused (no branch around it)
  const int kend = c0 + 16 * CB;
  XBuf x0, x1;
  fetch_x(0, x0);
  for (int k0 = 0; k0 < kend; k0 += 32) {
    step(k0, x0, k0 + 16, x1);
    step(k0 + 16, x1, min(k0 + 32, kend - 16), x0);
  }
#pragma unroll
  for (int ra = 0; ra < 4; ++ra)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = rb + 16 * ra + 4 * v + k;
      if (r < rows)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
          Y[(static_cast<int64_t>(t.a) + r) * RK + c0 + 16 * cb + i] = static_cast<float>(acc[ra][cb][v]);
    }
}

template <int RK>
__global__ __launch_bounds__(kBlock, RK >= kApplyMfmaRank ? 2 : 1) void k_apply(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  const MatDesc d = a.mats[t.idx];
  if constexpr (RK >= kApplyMfmaRank) {
    apply_mfma<RK>(a, t, d);
  } else {
    // W (upper triangular) is read at wave-uniform addresses, through the scalar cache into
    // SGPRs: every product takes its W entry from there rather than from an LDS broadcast
    const double* __restrict__ W = a.w + d.w_slot;
    {
      const int64_t row = static_cast<int64_t>(t.a) + tid();
      if (tid() >= t.b) return;
      const bool q = a.variant == 1;
      const float* X = a.fac + (q ? d.q_slot : d.p_slot) + row * RK;
      float* Y = a.fac + (q ? d.qh_slot : d.ph_slot) + row * RK;
      double x[RK];
      float y[RK];
      if constexpr (RK % 4 == 0) {  // factor slots are 256-byte aligned: rows are 16-byte aligned
#pragma unroll
        for (int l = 0; l < RK; l += 4) {
          const float4 v = *reinterpret_cast<const float4*>(X + l);
          x[l] = v.x;
          x[l + 1] = v.y;
          x[l + 2] = v.z;
          x[l + 3] = v.w;
        }
      } else {
#pragma unroll
        for (int l = 0; l < RK; ++l) x[l] = static_cast<double>(X[l]);
      }
      // y[k] = sum over l <= k of x[l] W[l][k], added in increasing l; by rows of W, each
      // row's entries loaded together
      double acc[RK];
#pragma unroll
      for (int k = 0; k < RK; ++k) acc[k] = 0.0;
#pragma unroll
      for (int l = 0; l < RK; ++l)
#pragma unroll
        for (int k = l; k < RK; ++k) acc[k] = fma(x[l], W[l * RK + k], acc[k]);
#pragma unroll
      for (int k = 0; k < RK; ++k) y[k] = static_cast<float>(acc[k]);
      if constexpr (RK % 4 == 0) {
#pragma unroll
        for (int k = 0; k < RK; k += 4)
          *reinterpret_cast<float4*>(Y + k) = make_float4(y[k], y[k + 1], y[k + 2], y[k + 3]);
      } else {
#pragma unroll
        for (int k = 0; k < RK; ++k) Y[k] = y[k];
      }
    }
  }
}

// ---------------------------------------------------------------------------------------
// Small rank-4 matrices whose rows are not 16-byte aligned (T_SMALL: n <= kSmallRows,
// m <= kSmallCols): one workgroup takes the whole matrix with scalar column accesses, inside
// the P-step, Q-step and decompress launches of the register-resident kernels.

// P-step: Qh = Q W (stored), per row P = M' Qh with M' = M + E (or M + F - Ph_row Q_loc^T),
// E = M' - P Qh^T, P to the factor buffer.  Shared memory: Wsh (16 doubles), qhs and qls
// (kSmallCols float4 each).
__device__ inline void small_pstep(const KArgs& a, const MatDesc& d, double* Wsh, float4* qhs, float4* qls) {
  const int n = d.n, m = d.m;
  const bool deferred = deferred_of(a, d.bucket);
  if (tid() < 16) Wsh[tid()] = a.w[d.w_slot + tid()];
  __syncthreads();
  const float4* Q4 = reinterpret_cast<const float4*>(a.fac + d.q_slot);
  const float4* Ql4 = reinterpret_cast<const float4*>(a.fac + d.ql_slot);
  float4* Qh4 = reinterpret_cast<float4*>(a.fac + d.qh_slot);
  for (int j = tid(); j < m; j += kBlock) {
    const float4 q = apply_w4(Q4[j], Wsh);
    qhs[j] = q;
    Qh4[j] = q;
    qls[j] = deferred ? Ql4[j] : zero4();
  }
  __syncthreads();
  const float* G = src_of(a, d.bucket) + d.grad_off;
  float* E = a.e + d.e_off;
  const float4* Ph4 = reinterpret_cast<const float4*>(a.fac + d.ph_slot);
  float* P = dst_of(a, d.bucket) + d.fac_off_p;
  const int wave = tid() >> 6, lane = tid() & 63;
  for (int row = wave; row < n; row += kBlock / kWave) {
    const float4 ph = deferred ? Ph4[row] : zero4();
    const int64_t base = static_cast<int64_t>(row) * m;
    auto mprime = [&](int j) {
      const float e = a.ef ? E[base + j] : 0.f;
      return (G[base + j] + e) - dot4(ph, qls[j]);
    };
    float4 acc = zero4();
    for (int j = lane; j < m; j += kWave) acc = fma4(mprime(j), qhs[j], acc);
    const float4 pr = wave_sum_dpp(acc);
    if (a.ef)
      for (int j = lane; j < m; j += kWave) E[base + j] = mprime(j) - dot4(pr, qhs[j]);
    if (lane < 4) P[static_cast<int64_t>(row) * 4 + lane] = lane == 0 ? pr.x : lane == 1 ? pr.y : lane == 2 ? pr.z : pr.w;
  }
}

// Q-step: Ph = P W (stored), F = M + E written back, Q_loc = F^T Ph summed over the rows in
// order, written to the factor buffer and the Ql slot (no row-chunk partials).  Shared memory:
// Wsh (16 doubles), phs (kSmallRows float4).
__device__ inline void small_qstep(const KArgs& a, const MatDesc& d, double* Wsh, float4* phs) {
  const int n = d.n, m = d.m;
  if (tid() < 16) Wsh[tid()] = a.w[d.w_slot + tid()];
  __syncthreads();
  const float4* P4 = reinterpret_cast<const float4*>(a.fac + d.p_slot);
  float4* Ph4 = reinterpret_cast<float4*>(a.fac + d.ph_slot);
  for (int i = tid(); i < n; i += kBlock) {
    const float4 y = apply_w4(P4[i], Wsh);
    phs[i] = y;
    Ph4[i] = y;
  }
  __syncthreads();
  const float* G = src_of(a, d.bucket) + d.grad_off;
  float* E = a.e + d.e_off;
  float* Q = dst_of(a, d.bucket) + d.fac_off_q;
  float* Ql = a.fac + d.ql_slot;
  for (int j = tid(); j < m; j += kBlock) {
    float4 acc = zero4();
    for (int row = 0; row < n; ++row) {
      const int64_t idx = static_cast<int64_t>(row) * m + j;
      float f = G[idx];
      if (a.ef) {
        f += E[idx];
        E[idx] = f;
      }
      acc = fma4(f, phs[row], acc);
    }
    const float q[4] = {acc.x, acc.y, acc.z, acc.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      Q[static_cast<int64_t>(j) * 4 + k] = q[k];
      Ql[static_cast<int64_t>(j) * 4 + k] = q[k];
    }
  }
}

// Decompress: M_hat = A B^T / p (odd step: A = P_agg, B = Qh; even step: A = Ph, B = Q_agg).
// Shared memory: bs (kSmallCols float4).
__device__ inline void small_recon(const KArgs& a, const MatDesc& d, float4* bs) {
  const int n = d.n, m = d.m;
  const bool odd = a.parity != 0;
  const float* agg = src_of(a, d.bucket);
  const float* A = odd ? agg + d.fac_off_p : a.fac + d.ph_slot;
  const float* B = odd ? a.fac + d.qh_slot : agg + d.fac_off_q;
  for (int j = tid(); j < m; j += kBlock)
    bs[j] = make_float4(B[4 * j], B[4 * j + 1], B[4 * j + 2], B[4 * j + 3]);
  __syncthreads();
  float* O = dst_of(a, d.bucket) + d.grad_off;
  const int wave = tid() >> 6, lane = tid() & 63;
  for (int row = wave; row < n; row += kBlock / kWave) {
    const float* ar = A + static_cast<int64_t>(row) * 4;
    const float4 av = scale4(make_float4(ar[0], ar[1], ar[2], ar[3]), a.inv_p);
    for (int j = lane; j < m; j += kWave) O[static_cast<int64_t>(row) * m + j] = dot4(av, bs[j]);
  }
}

// ---------------------------------------------------------------------------------------
// Narrow rows (r = 4, 16-byte aligned rows of at most 512 columns): L lanes per row (16, 32 or
// 64), G float4 groups per lane (1 or 2).  A wave holds 64 / L whole rows at a time and the
// workgroup 256 / L; lane l of row slot l / L owns groups (l % L) + L g, whose factor rows stay
// in registers.  Row sums stay inside the wave, so these kernels wait at no barrier per row.
template <int L, int G>
struct Narrow {
  static constexpr int SL = 64 / L;   // rows per wave at a time
  static constexpr int RW = 4 * SL;   // rows per workgroup round
  int wave, slot, cl;
  int c4[G];
  bool ok[G];
  __device__ explicit Narrow(int m4) {
    wave = __builtin_amdgcn_readfirstlane(tid() >> 6);
    const int lane = tid() & 63;
    slot = lane / L;
    cl = lane % L;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      c4[g] = cl + L * g;
      ok[g] = c4[g] < m4;
    }
  }
  __device__ int row(int k) const { return k * RW + wave * SL + slot; }  // tile-relative row of round k
};

// Sum over the L lanes of a row slot; every lane of the slot gets the same bits.  DPP quad
// butterflies and mirrors give 16-lane sums, a swizzle (xor 16) pairs them for L = 32, and for
// L = 64 the four 16-lane sums are read out and added in order.
template <int L>
__device__ inline float row_sum(float v) {
  v += dpp<0xB1>(v);
  v += dpp<0x4E>(v);
  v += dpp<0x141>(v);
  v += dpp<0x140>(v);
  if constexpr (L == 32)
    v += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x401F));
  if constexpr (L == 64) {
    const int b = __builtin_bit_cast(int, v);
    v = ((__builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 0)) +
          __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 16))) +
         __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 32))) +
        __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 48));
  }
  return v;
}
template <int L>
__device__ inline float4 row_sum4(const float4& v) {
  return make_float4(row_sum<L>(v.x), row_sum<L>(v.y), row_sum<L>(v.z), row_sum<L>(v.w));
}

// The lane's Qh rows (Q W) and Q_loc rows for its columns; the tile holding row 0 stores Qh.
template <int L, int G>
__device__ inline void narrow_qfactors(const KArgs& a, const MatDesc& d, const Narrow<L, G>& nm,
                                       const double* Wsh, bool store_qh, bool deferred,
                                       float4 (&qh)[G][4], float4 (&ql)[G][4]) {
  const float4* Q4 = reinterpret_cast<const float4*>(a.fac + d.q_slot);
  const float4* Ql4 = reinterpret_cast<const float4*>(a.fac + d.ql_slot);
  float4* Qh4 = reinterpret_cast<float4*>(a.fac + d.qh_slot);
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int j = 4 * (nm.ok[g] ? nm.c4[g] : 0) + c;  // in-range row for lanes past m
      const float4 q = apply_w4(Q4[j], Wsh);
      const float4 l = Ql4[j];
      qh[g][c] = nm.ok[g] ? q : zero4();
      ql[g][c] = (nm.ok[g] && deferred) ? l : zero4();
      if (store_qh && nm.ok[g]) Qh4[j] = q;
    }
}

// P-step, narrow rows: per row M' = M + E (or M + F - Ph_row Q_loc^T), P = M' Qh (row sum),
// E = M' - P Qh^T, P to the factor buffer.  U rounds of rows are in flight per lane.  Wsh: 16
// doubles of shared memory.
template <int L, int G>
__device__ void pnarrow_tile(const KArgs& a, const Tile& t, const MatDesc& d, double* Wsh) {
  using NM = Narrow<L, G>;
  constexpr int U = 2;
  const NM nm(d.m >> 2);
  const bool deferred = deferred_of(a, d.bucket);
  const uint32_t row_bytes = static_cast<uint32_t>(d.m) * 4u;
  const uint32_t tile_bytes = static_cast<uint32_t>(t.b) * row_bytes;
  const int64_t first = static_cast<int64_t>(t.a) * d.m;
  const Rsrc Gr = tile_rsrc(src_of(a, d.bucket) + d.grad_off + first, tile_bytes);
  const Rsrc Er = tile_rsrc(a.e + d.e_off + first, a.ef ? tile_bytes : 0u);
  const Rsrc Pr = tile_rsrc(dst_of(a, d.bucket) + d.fac_off_p + static_cast<int64_t>(t.a) * 4,
                            static_cast<uint32_t>(t.b) * 16u);
  const Rsrc Phr = tile_rsrc(a.fac + d.ph_slot + static_cast<int64_t>(t.a) * 4,
                             deferred ? static_cast<uint32_t>(t.b) * 16u : 0u);
  uint32_t coff[G];
#pragma unroll
  for (int g = 0; g < G; ++g) coff[g] = nm.ok[g] ? static_cast<uint32_t>(nm.c4[g]) * 16u : kOut;

  float4 gv[U][G], ev[U][G], ph[U];
  auto load = [&](int k0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t row = static_cast<uint32_t>(nm.row(k0 + u));  // past the tile: zeros
      const uint32_t roff = row * row_bytes;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const uint32_t o = coff[g] == kOut ? kOut : roff + coff[g];
        gv[u][g] = bld4_nt(Gr, o);
        ev[u][g] = bld4_nt(Er, o);
      }
      ph[u] = bld4(Phr, row * 16u);
    }
  };
  load(0);
  if (tid() < 16) Wsh[tid()] = a.w[d.w_slot + tid()];
  __syncthreads();
  float4 qh[G][4], ql[G][4];
  narrow_qfactors(a, d, nm, Wsh, t.a == 0 && nm.wave == 0 && nm.slot == 0, deferred, qh, ql);

  for (int k = 0; k * NM::RW < t.b; k += U) {
    float4 mp[U][G], acc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      acc[u] = zero4();
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float4 v = gv[u][g] + ev[u][g];
        v.x -= dot4(ph[u], ql[g][0]);
        v.y -= dot4(ph[u], ql[g][1]);
        v.z -= dot4(ph[u], ql[g][2]);
        v.w -= dot4(ph[u], ql[g][3]);
        mp[u][g] = v;
        acc[u] = fma4(v.x, qh[g][0], acc[u]);
        acc[u] = fma4(v.y, qh[g][1], acc[u]);
        acc[u] = fma4(v.z, qh[g][2], acc[u]);
        acc[u] = fma4(v.w, qh[g][3], acc[u]);
      }
    }
    load(k + U);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float4 P = row_sum4<L>(acc[u]);
      const uint32_t row = static_cast<uint32_t>(nm.row(k + u));
      const uint32_t roff = row * row_bytes;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float4 r = mp[u][g];
        r.x -= dot4(P, qh[g][0]);
        r.y -= dot4(P, qh[g][1]);
        r.z -= dot4(P, qh[g][2]);
        r.w -= dot4(P, qh[g][3]);
        bst4_nt(Er, coff[g] == kOut ? kOut : roff + coff[g], r);
      }
      bst4(Pr, nm.cl == 0 ? row * 16u : kOut, P);
    }
  }
}

// Q-step, narrow rows (r = 4, fused orthogonalisation): tile = row chunk t.a.  The chunk's Ph
// rows are formed in LDS as P W (and stored to the Ph slot); per row F = M + E is written back
// and each lane adds F^T Ph over its rows and columns.  The 256 / L row slots' sums are added in
// slot order through LDS and stored as the chunk's partials for K_QFIN.  Shared memory: Wsh (16
// doubles), phs (kQRows float4), red (kNarrowRed float4).
constexpr int kNarrowRed = 2048;  // float4: row slots x L G 4 at most (4 x 64 x 2 x 4)
template <int L, int G>
__device__ void qnarrow_tile(const KArgs& a, const Tile& t, const MatDesc& d, double* Wsh, float4* phs,
                             float4* red) {
  using NM = Narrow<L, G>;
  constexpr int U = 2;
  constexpr int NS = 4 * NM::SL;  // row slots of the workgroup
  static_assert(NS * L * G * 4 <= kNarrowRed, "slot sums exceed the shared buffer");
  const int m4 = d.m >> 2;
  const NM nm(m4);
  const int64_t r0 = static_cast<int64_t>(t.a) * d.q_rows;
  const int rows = static_cast<int>((r0 + d.q_rows < d.n) ? d.q_rows : d.n - r0);
  const uint32_t row_bytes = static_cast<uint32_t>(d.m) * 4u;
  const uint32_t ext = static_cast<uint32_t>(rows) * row_bytes;
  const int64_t first = r0 * d.m;
  const Rsrc Gr = tile_rsrc(src_of(a, d.bucket) + d.grad_off + first, ext);
  const Rsrc Er = tile_rsrc(a.e + d.e_off + first, a.ef ? ext : 0u);
  uint32_t coff[G];
#pragma unroll
  for (int g = 0; g < G; ++g) coff[g] = nm.ok[g] ? static_cast<uint32_t>(nm.c4[g]) * 16u : kOut;

  float4 gv[U][G], ev[U][G];
  auto load = [&](int k0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t roff = static_cast<uint32_t>(nm.row(k0 + u)) * row_bytes;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const uint32_t o = coff[g] == kOut ? kOut : roff + coff[g];
        gv[u][g] = bld4_nt(Gr, o);
        ev[u][g] = bld4_nt(Er, o);
      }
    }
  };
  load(0);
  if (tid() < 16) Wsh[tid()] = a.w[d.w_slot + tid()];
  __syncthreads();
  if (tid() < kQRows) {
    float4 y = zero4();
    if (tid() < rows) {
      const int64_t row = r0 + tid();
      y = apply_w4(reinterpret_cast<const float4*>(a.fac + d.p_slot)[row], Wsh);
      reinterpret_cast<float4*>(a.fac + d.ph_slot)[row] = y;
    }
    phs[tid()] = y;
  }
  __syncthreads();

  float4 acc[G][4];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[g][c] = zero4();
  for (int k = 0; k * NM::RW < rows; k += U) {
    float4 f[U][G];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int g = 0; g < G; ++g) f[u][g] = gv[u][g] + ev[u][g];
    load(k + U);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int row = nm.row(k + u);  // < kQRows: rows <= kQRows and 2 RW divides kQRows
      const uint32_t roff = static_cast<uint32_t>(row) * row_bytes;
      const float4 ph = phs[row & (kQRows - 1)];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        bst4_nt(Er, coff[g] == kOut ? kOut : roff + coff[g], f[u][g]);
        acc[g][0] = fma4(f[u][g].x, ph, acc[g][0]);
        acc[g][1] = fma4(f[u][g].y, ph, acc[g][1]);
        acc[g][2] = fma4(f[u][g].z, ph, acc[g][2]);
        acc[g][3] = fma4(f[u][g].w, ph, acc[g][3]);
      }
    }
  }
  const int sidx = nm.wave * NM::SL + nm.slot;
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int c = 0; c < 4; ++c) red[sidx * (L * G * 4) + (nm.cl * G + g) * 4 + c] = acc[g][c];
  __syncthreads();
  const int64_t ncb = (d.m + d.q_cb - 1) / d.q_cb;
  float4* part = reinterpret_cast<float4*>(a.qpart + d.qpart + static_cast<int64_t>(t.a) * ncb * d.q_cb * 4);
  for (int e = tid(); e < L * G * 4; e += kBlock) {
    const int cl = e / (G * 4), g = (e / 4) % G, c = e % 4;
    const int col4 = cl + L * g;
    if (col4 >= m4) continue;
    float4 sum = red[e];
    for (int sl = 1; sl < NS; ++sl) sum = sum + red[sl * (L * G * 4) + e];
    part[4 * col4 + c] = sum;  // Q partial of column 4 col4 + c, ranks 0..3
  }
}

// Decompress, narrow rows: M_hat rows from the tile's A rows (staged in LDS, scaled by 1 / p)
// and the lane's B rows in registers.  as: kMaxTileRows float4 of shared memory.
template <int L, int G>
__device__ void rnarrow_tile(const KArgs& a, const Tile& t, const MatDesc& d, float4* as) {
  using NM = Narrow<L, G>;
  const bool odd = a.parity != 0;
  const NM nm(d.m >> 2);
  const float* agg = src_of(a, d.bucket);
  const float4* A4 = reinterpret_cast<const float4*>(odd ? agg + d.fac_off_p : a.fac + d.ph_slot);
  const float4* B4 = reinterpret_cast<const float4*>(odd ? a.fac + d.qh_slot : agg + d.fac_off_q);
  if (tid() < t.b) as[tid()] = scale4(A4[t.a + tid()], a.inv_p);  // the tile's A rows / p
  float4 b[G][4];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int c = 0; c < 4; ++c) b[g][c] = nm.ok[g] ? B4[4 * nm.c4[g] + c] : zero4();
  __syncthreads();
  __builtin_amdgcn_s_waitcnt(0);
  const uint32_t row_bytes = static_cast<uint32_t>(d.m) * 4u;
  const Rsrc O = tile_rsrc(dst_of(a, d.bucket) + d.grad_off + static_cast<int64_t>(t.a) * d.m,
                           static_cast<uint32_t>(t.b) * row_bytes);
  uint32_t coff[G];
#pragma unroll
  for (int g = 0; g < G; ++g) coff[g] = nm.ok[g] ? static_cast<uint32_t>(nm.c4[g]) * 16u : kOut;
  for (int k = 0; k * NM::RW < t.b; ++k) {
    const int row = nm.row(k);  // past the tile: an unset LDS entry, its stores are dropped
    const float4 ar = as[row & (kMaxTileRows - 1)];
    const uint32_t roff = static_cast<uint32_t>(row) * row_bytes;
#pragma unroll
    for (int g = 0; g < G; ++g)
      bst4_nt(O, coff[g] == kOut ? kOut : roff + coff[g],
           make_float4(dot4(ar, b[g][0]), dot4(ar, b[g][1]), dot4(ar, b[g][2]), dot4(ar, b[g][3])));
  }
}

// Narrow-row tiles of a matrix (at most 128 float4 groups per row) inside the rank-4 P-step,
// Q-step and decompress launches: the variant follows from the row length.
__device__ inline void narrow_pstep(const KArgs& a, const Tile& t, const MatDesc& d, double* Wsh) {
  switch (narrow_variant(d.m >> 2)) {
    case (16 << 4) | 1: pnarrow_tile<16, 1>(a, t, d, Wsh); break;
    case (32 << 4) | 1: pnarrow_tile<32, 1>(a, t, d, Wsh); break;
    case (64 << 4) | 1: pnarrow_tile<64, 1>(a, t, d, Wsh); break;
    default: pnarrow_tile<64, 2>(a, t, d, Wsh); break;
  }
}
__device__ inline void narrow_qstep(const KArgs& a, const Tile& t, const MatDesc& d, double* Wsh,
                                    float4* phs, float4* red) {
  switch (narrow_variant(d.m >> 2)) {
    case (16 << 4) | 1: qnarrow_tile<16, 1>(a, t, d, Wsh, phs, red); break;
    case (32 << 4) | 1: qnarrow_tile<32, 1>(a, t, d, Wsh, phs, red); break;
    case (64 << 4) | 1: qnarrow_tile<64, 1>(a, t, d, Wsh, phs, red); break;
    default: qnarrow_tile<64, 2>(a, t, d, Wsh, phs, red); break;
  }
}
__device__ inline void narrow_recon(const KArgs& a, const Tile& t, const MatDesc& d, float4* as) {
  switch (narrow_variant(d.m >> 2)) {
    case (16 << 4) | 1: rnarrow_tile<16, 1>(a, t, d, as); break;
    case (32 << 4) | 1: rnarrow_tile<32, 1>(a, t, d, as); break;
    case (64 << 4) | 1: rnarrow_tile<64, 1>(a, t, d, as); break;
    default: rnarrow_tile<64, 2>(a, t, d, as); break;
  }
}

// ---------------------------------------------------------------------------------------
// Column mapping shared by the rank-4 streaming kernels.  The W waves of a workgroup (four, or
// three for rows of at most 768 columns) split a row of m4 = m / 4 float4 groups into W
// segments of 64 Se groups, Se = ceil(m4 / 64 W) <= S
// (a launch of class S also carries rows of smaller classes); lane `lane` of wave w owns groups
// w * 64 Se + s * 64 + lane, s < Se, for every row of the tile, so the factor rows of those
// columns are loaded once per workgroup and kept in registers.  The waves work on the same RB
// rows at a time (8 for S = 1, 2 for S = 2..4, 1 for S = 5).
template <int S, int W = 4>
struct Cols {
  static constexpr int RB = S == 1 ? 8 : (S <= 4 ? 2 : 1);
  int wave, lane;
  int c4[S];
  bool ok[S];
  __device__ explicit Cols(int m4) {
    wave = tid() >> 6;
    lane = tid() & 63;
    const int se = (m4 + 64 * W - 1) / (64 * W);
#pragma unroll
    for (int s = 0; s < S; ++s) {
      c4[s] = wave * 64 * se + s * 64 + lane;
      ok[s] = s < se && c4[s] < m4;
    }
  }
};

// P-step, fused single pass (r = 4, 16-byte aligned rows of up to 5120 columns).  Each lane
// keeps, for its columns, the rows of Qh = Q W (computed here from the reused factor; the tile
// holding row 0 also stores Qh) and of Q_loc in registers for the whole tile (Q_loc and the
// tile's Ph rows are zero unless E is deferred).  Per row: M' = M + E (or M + F - Ph_row
// Q_loc^T), P = M' Qh summed over the row (DPP wave sums, then the four waves' sums in wave
// order), E = M' - P Qh^T written back, P written to the factor buffer.  The next rows' M and
// E are requested before the reduction; all streamed accesses are tile-relative buffer
// accesses (E's resource is empty when error feedback is off).
template <int S, int W = 4>
__global__ __launch_bounds__(64 * W) void k_pfused(KArgs a) {
  constexpr int RB = Cols<S, W>::RB;
  const Tile t = a.tiles[blockIdx.x];
  if (t.kind == T_VEC) {
    vec_tile(a, t, true);
    return;
  }
  const MatDesc d = a.mats[t.idx];
  if constexpr (S == 1 && W == 4) {
    if (t.kind == T_ROWS) {  // a narrow-row matrix's tile (the S = 1 launch carries them)
      __shared__ double Wn[16];
      narrow_pstep(a, t, d, Wn);
      return;
    }
    if (t.kind == T_SMALL) {  // a small matrix, whole (the S = 1 launch carries them)
      __shared__ double Ws[16];
      __shared__ float4 qhs[kSmallCols], qls[kSmallCols];
      small_pstep(a, d, Ws, qhs, qls);
      return;
    }
  }
  const int m4 = d.m >> 2;
  const Cols<S, W> cl(m4);
  const bool deferred = deferred_of(a, d.bucket);
  // tile rows t.a + k * stride, k < rows (T_SROWS)
  const int stride = (t.b >> 4) & 0xfff, rows = t.b >> 16;
  const uint32_t row_bytes = static_cast<uint32_t>(d.m) * 4u;
  const uint32_t step_bytes = static_cast<uint32_t>(stride) * row_bytes;
  const uint32_t tile_bytes = static_cast<uint32_t>(rows - 1) * step_bytes + row_bytes;
  const int64_t first = static_cast<int64_t>(t.a) * d.m;
  const Rsrc G = tile_rsrc(src_of(a, d.bucket) + d.grad_off + first, tile_bytes);
  const Rsrc E = tile_rsrc(a.e + d.e_off + first, a.ef ? tile_bytes : 0u);
  const Rsrc P = tile_rsrc(dst_of(a, d.bucket) + d.fac_off_p + static_cast<int64_t>(t.a) * 4,
                           static_cast<uint32_t>((rows - 1) * stride + 1) * 16u);
  uint32_t coff[S];
#pragma unroll
  for (int s = 0; s < S; ++s) coff[s] = cl.ok[s] ? static_cast<uint32_t>(cl.c4[s]) * 16u : kOut;

  // the first rows' M and E are requested before the factor setup
  float4 g[RB][S], e[RB][S];
  auto load_rows = [&](int r0) {  // tile-relative first row
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int s = 0; s < S; ++s) {
        const uint32_t o = static_cast<uint32_t>(r0 + rb) * step_bytes + coff[s];
        g[rb][s] = bld4_nt(G, o);
        e[rb][s] = bld4_nt(E, o);
      }
  };
  load_rows(0);

  __shared__ double Wsh[16];
  __shared__ float4 red[2][W][RB];
  __shared__ float4 phs[kMaxTileRows];  // the tile's rows of Ph (zero unless E is deferred)
  if (tid() < 16) Wsh[tid()] = a.w[d.w_slot + tid()];
  for (int i = tid(); i < rows; i += 64 * W)
    phs[i] = deferred ? reinterpret_cast<const float4*>(a.fac + d.ph_slot)[t.a + static_cast<int64_t>(i) * stride]
                      : zero4();
  __syncthreads();

  const float4* Q4 = reinterpret_cast<const float4*>(a.fac + d.q_slot);
  const float4* Ql4 = reinterpret_cast<const float4*>(a.fac + d.ql_slot);
  float4* Qh4 = reinterpret_cast<float4*>(a.fac + d.qh_slot);
  const bool store_qh = t.a == 0;
  float4 qh[S][4], ql[S][4];
#pragma unroll
  for (int s = 0; s < S; ++s)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int j = 4 * (cl.ok[s] ? cl.c4[s] : 0) + c;  // in-range row for lanes past m
      const float4 q = apply_w4(Q4[j], Wsh);
      const float4 l = Ql4[j];
      qh[s][c] = cl.ok[s] ? q : zero4();
      ql[s][c] = (cl.ok[s] && deferred) ? l : zero4();
      if (store_qh && cl.ok[s]) Qh4[j] = q;
    }

  int buf = 0;
  for (int r0 = 0; r0 < rows; r0 += RB, buf ^= 1) {
    float4 mp[RB][S];
    float4 acc[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      // rows past the tile read phs entries that are never used: their stores are dropped
      const float4 ph = phs[(r0 + rb) & (kMaxTileRows - 1)];
      acc[rb] = zero4();
#pragma unroll
      for (int s = 0; s < S; ++s) {
        float4 v = g[rb][s] + e[rb][s];
        v.x -= dot4(ph, ql[s][0]);
        v.y -= dot4(ph, ql[s][1]);
        v.z -= dot4(ph, ql[s][2]);
        v.w -= dot4(ph, ql[s][3]);
        mp[rb][s] = v;
        acc[rb] = fma4(v.x, qh[s][0], acc[rb]);
        acc[rb] = fma4(v.y, qh[s][1], acc[rb]);
        acc[rb] = fma4(v.z, qh[s][2], acc[rb]);
        acc[rb] = fma4(v.w, qh[s][3], acc[rb]);
      }
    }
    load_rows(r0 + RB);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      acc[rb] = wave_sum_dpp(acc[rb]);
      if (cl.lane == 0) red[buf][cl.wave][rb] = acc[rb];
    }
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const uint32_t roff = static_cast<uint32_t>(r0 + rb) * step_bytes;
      float4 Pr = red[buf][0][rb];  // the waves' sums in wave order
#pragma unroll
      for (int w = 1; w < W; ++w) Pr = Pr + red[buf][w][rb];
#pragma unroll
      for (int s = 0; s < S; ++s) {
        float4 r = mp[rb][s];
        r.x -= dot4(Pr, qh[s][0]);
        r.y -= dot4(Pr, qh[s][1]);
        r.z -= dot4(Pr, qh[s][2]);
        r.w -= dot4(Pr, qh[s][3]);
        bst4_nt(E, roff + coff[s], r);
      }
      bst4(P, tid() == 0 ? static_cast<uint32_t>((r0 + rb) * stride) * 16u : kOut, Pr);
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
  const float* G = src_of(a, d.bucket) + d.grad_off + row * m;
  const float* E = a.e + d.e_off + row * m;
  const float* Qh = a.fac + d.qh_slot;
  const float* Ql = a.fac + d.ql_slot;
  const bool ef = a.ef != 0, deferred = deferred_of(a, d.bucket);
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
    dst_of(a, d.bucket)[d.fac_off_p + row * RK + k] = ((red[0][k] + red[1][k]) + red[2][k]) + red[3][k];
  }
}

// P-step, general: E = M' - P Qh^T over a tile of rows (P from the factor buffer).
template <int RK>
__global__ __launch_bounds__(kBlock) void k_eupd(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  const MatDesc d = a.mats[t.idx];
  const int64_t m = d.m;
  const bool deferred = deferred_of(a, d.bucket);
  const float* Qh = a.fac + d.qh_slot;
  const float* Ql = a.fac + d.ql_slot;
  const float* Ph = a.fac + d.ph_slot;
  const float* P = dst_of(a, d.bucket) + d.fac_off_p;
  const float* G = src_of(a, d.bucket) + d.grad_off;
  const int64_t total = static_cast<int64_t>(t.b) * m;
  for (int64_t e = tid(); e < total; e += kBlock) {
    const int64_t row = t.a + e / m, j = e % m;
    const int64_t idx = row * m + j;
    float mp = G[idx] + a.e[d.e_off + idx];
    if (deferred)
#pragma unroll
      for (int k = 0; k < RK; ++k) mp -= Ph[row * RK + k] * Ql[j * RK + k];
    float r = mp;
#pragma unroll
    for (int k = 0; k < RK; ++k) r -= P[row * RK + k] * Qh[j * RK + k];
    a.e[d.e_off + idx] = r;
  }
}

// Write E of a tile of rows into a bucket-shaped output: the arena itself, F - Ph Q_loc^T
// (after a Q-step) or X - P_loc Qh^T (after a P-step of rank >= 8).
template <int RK>
__global__ __launch_bounds__(kBlock) void k_emat(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  const MatDesc d = a.mats[t.idx];
  const int64_t m = d.m;
  const bool fform = deferred_of(a, d.bucket), xform = deferred_p_of(a, d.bucket);
  const float* L = a.fac + (xform ? d.qh_slot : d.ql_slot);  // column factor of the term
  const float* R = a.fac + (xform ? d.pl_slot : d.ph_slot);  // row factor of the term
  float* out = dst_of(a, d.bucket);
  const int64_t total = static_cast<int64_t>(t.b) * m;
  for (int64_t e = tid(); e < total; e += kBlock) {
    const int64_t row = t.a + e / m, j = e % m;
    const int64_t idx = row * m + j;
    float v = a.e[d.e_off + idx];
    if (fform || xform)
#pragma unroll
      for (int k = 0; k < RK; ++k) v -= R[row * RK + k] * L[j * RK + k];
    out[d.grad_off + idx] = v;
  }
}

// ---------------------------------------------------------------------------------------
// Q-step: tile = (row chunk of at most kQRows rows, column block of 4 x 64 x CPT columns).
// Wave w owns the CPT adjacent columns cb * q_cb + (w * 64 + lane) * CPT of every row of the
// chunk, so each row's 4 KB (CPT = 4) segment is read by one workgroup.  The chunk's Ph rows are
// staged in LDS first (FUSED, r = 4: formed here as P W, and stored by the tiles of column
// block 0).  Per row: F = M' = M + E written back (deferred E), partial Q += M'^T Ph over the
// lane's columns.  Rows go in groups of U whose loads are issued before the previous group's
// F stores, so stores never hold up the next loads.  Each lane stores its partial sums for
// K_QFIN (lanes past m store zeros into the padded partial block).
template <int RK, int CPT, bool FUSED>
__global__ __launch_bounds__(kBlock) void k_qstep(KArgs a) {
  constexpr int U = 8;  // rows per group
  using Vec = typename std::conditional<CPT == 4, float4, float>::type;
  const Tile t = a.tiles[blockIdx.x];
  if (t.kind == T_VEC) {
    vec_tile(a, t, true);
    return;
  }
  const MatDesc d = a.mats[t.idx];
  __shared__ double Wsh[16];
  __shared__ __align__(16) float phs[kQRows * RK];
  if constexpr (FUSED) {
    static_assert(kSmallRows <= kQRows, "a small matrix's Ph rows use the chunk's Ph buffer");
    if (t.kind == T_SMALL) {  // a small matrix, whole (the fused launch carries them)
      small_qstep(a, d, Wsh, reinterpret_cast<float4*>(phs));
      return;
    }
    if (d.scls == 0) {  // a narrow-row matrix's chunk (the fused launch carries them)
      __shared__ float4 red[kNarrowRed];
      narrow_qstep(a, t, d, Wsh, reinterpret_cast<float4*>(phs), red);
      return;
    }
  }
  const int wave = tid() >> 6, lane = tid() & 63;
  const int64_t m = d.m;
  const ChunkRows ch = q_chunk_rows(d, t.a);  // rows ch.first + k * ch.stride, k < ch.rows
  const int64_t r0 = ch.first;
  const int rows = ch.rows;
  const int64_t cb0 = static_cast<int64_t>(t.b) * d.q_cb;
  const int lcol = (wave * 64 + lane) * CPT;  // column within the block
  const int64_t bcols = (m - cb0) < d.q_cb ? (m - cb0) : d.q_cb;
  const bool valid = lcol < bcols;
  const uint32_t step_bytes = static_cast<uint32_t>(ch.stride) * static_cast<uint32_t>(m) * 4u;
  // extent from the block's first column of the chunk's first row to its last element
  const uint32_t ext = static_cast<uint32_t>(rows - 1) * step_bytes + static_cast<uint32_t>(bcols) * 4u;
  const int64_t first = r0 * m + cb0;
  const Rsrc G = tile_rsrc(src_of(a, d.bucket) + d.grad_off + first, ext);
  const Rsrc E = tile_rsrc(a.e + d.e_off + first, a.ef ? ext : 0u);
  const uint32_t coff = valid ? static_cast<uint32_t>(lcol) * 4u : kOut;

  Vec g[U], e[U];
  auto load_group = [&](int rr, Vec* gg, Vec* ee) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t o = static_cast<uint32_t>(rr + u) * step_bytes + coff;
      if constexpr (CPT == 4) {
        gg[u] = bld4_nt(G, o);
        ee[u] = bld4_nt(E, o);
      } else {
        gg[u] = bld1_nt(G, o);
        ee[u] = bld1_nt(E, o);
      }
    }
  };
  load_group(0, g, e);

  // the chunk's Ph rows; the rows after them are zero (groups may run past the chunk)
  static_assert(kQRows <= kBlock && kQRows % 8 == 0, "one thread per staged Ph row");
  if constexpr (FUSED) {
    if (tid() < 16) Wsh[tid()] = a.w[d.w_slot + tid()];
    __syncthreads();
    if (tid() < kQRows) {
      float4 y = zero4();
      if (tid() < rows) {
        const int64_t row = r0 + static_cast<int64_t>(tid()) * ch.stride;
        y = apply_w4(*reinterpret_cast<const float4*>(a.fac + d.p_slot + row * 4), Wsh);
        if (t.b == 0) *reinterpret_cast<float4*>(a.fac + d.ph_slot + row * 4) = y;
      }
      *reinterpret_cast<float4*>(&phs[tid() * 4]) = y;
    }
  } else {
    for (int i = tid(); i < kQRows * RK; i += kBlock)
      phs[i] = i < rows * RK ? a.fac[d.ph_slot + (r0 + static_cast<int64_t>(i / RK) * ch.stride) * RK + i % RK] : 0.f;
  }
  __syncthreads();

  float acc[CPT][RK];
#pragma unroll
  for (int c = 0; c < CPT; ++c)
#pragma unroll
    for (int k = 0; k < RK; ++k) acc[c][k] = 0.f;

  for (int rr = 0; rr < rows; rr += U) {
    Vec gn[U], en[U];
    load_group(rr + U, gn, en);
    Vec f[U];
#pragma unroll
    for (int u = 0; u < U; ++u) f[u] = g[u] + e[u];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t o = static_cast<uint32_t>(rr + u) * step_bytes + coff;
      if constexpr (CPT == 4)
        bst4_nt(E, o, f[u]);
      else
        bst1_nt(E, o, f[u]);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float* ph = &phs[(rr + u) * RK];  // rr + u < kQRows: kQRows is a multiple of U
      float mp[CPT];
      if constexpr (CPT == 4) {
        mp[0] = f[u].x;
        mp[1] = f[u].y;
        mp[2] = f[u].z;
        mp[3] = f[u].w;
      } else {
        mp[0] = f[u];
      }
#pragma unroll
      for (int c = 0; c < CPT; ++c)
#pragma unroll
        for (int k = 0; k < RK; ++k) acc[c][k] = fmaf(mp[c], ph[k], acc[c][k]);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      g[u] = gn[u];
      e[u] = en[u];
    }
  }
  const int64_t ncb = (m + d.q_cb - 1) / d.q_cb;
  const int64_t stride = ncb * d.q_cb * RK;  // one row chunk of partials
  float* part = a.qpart + d.qpart + static_cast<int64_t>(t.a) * stride + (cb0 + lcol) * RK;
#pragma unroll
  for (int c = 0; c < CPT; ++c)
#pragma unroll
    for (int k = 0; k < RK; ++k) part[c * RK + k] = acc[c][k];
}

// Q-step finish: Q_loc = sum over the row chunks' partials.  A tile covers the NE entries
// [t.a * NE, t.a * NE + NE) of the matrix (entry e = column * r + rank, NE = qfin_entries):
// with NE > 256 each thread takes NE / 256 entries 256 apart, otherwise 256 / NE threads share
// an entry.  Each thread adds a contiguous share of the chunks in chunk order, eight chunks
// requested at a time, and the shares are added in thread order.  The result goes to the factor
// buffer and to the Ql slot.
template <int RK>
__global__ __launch_bounds__(kBlock) void k_qfin(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  if (t.kind == T_VEC) {  // from kWideRank on the finish launch packs the raw vectors too
    vec_tile(a, t, true);
    return;
  }
  const MatDesc d = a.mats[t.idx];
  const int64_t m = d.m;
  const int64_t ncb = (m + d.q_cb - 1) / d.q_cb;
  const int64_t stride = ncb * d.q_cb * RK;  // one row chunk of partials
  const int ne = qfin_entries(d.q_chunks);   // entries per tile
  const float* part = a.qpart + d.qpart;
  float* out = dst_of(a, d.bucket) + d.fac_off_q;
  float* ql = a.fac + d.ql_slot;
  constexpr int U = 8;
  if (ne > kBlock) {  // at most 8 chunks: one thread per entry
    constexpr int EPT = 4;  // entries per thread (ne = 1024)
    float s[EPT];
    int64_t e[EPT];
#pragma unroll
    for (int k = 0; k < EPT; ++k) {
      e[k] = static_cast<int64_t>(t.a) * ne + tid() + k * kBlock;
      s[k] = 0.f;
    }
    {
      // all (at most 8) chunks of the thread's entries requested together, added in chunk order
      float v[EPT][8];
#pragma unroll
      for (int k = 0; k < EPT; ++k)
#pragma unroll
        for (int u = 0; u < 8; ++u)
          v[k][u] = (e[k] < m * RK && u < d.q_chunks) ? part[u * stride + e[k]] : 0.f;
#pragma unroll
      for (int k = 0; k < EPT; ++k)
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (u < d.q_chunks) s[k] += v[k][u];
    }
#pragma unroll
    for (int k = 0; k < EPT; ++k)
      if (e[k] < m * RK) {
        out[e[k]] = s[k];
        ql[e[k]] = s[k];
      }
    return;
  }
  const int ng = kBlock / ne;                // threads per entry
  const int gq = tid() / ne, el = tid() % ne;
  const int64_t e = static_cast<int64_t>(t.a) * ne + el;
  const bool on = e < m * RK;
  const int per = (d.q_chunks + ng - 1) / ng;
  const int ch0 = gq * per, ch1 = (ch0 + per < d.q_chunks) ? ch0 + per : d.q_chunks;
  float s = 0.f;
  if (on) {
    const float* base = part + e;
    int ch = ch0;
    for (; ch + U <= ch1; ch += U) {
      float v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = base[(ch + u) * stride];
#pragma unroll
      for (int u = 0; u < U; ++u) s += v[u];
    }
    if (ch < ch1) {  // the rest (fewer than U chunks) requested together too, added in order
      float v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = ch + u < ch1 ? base[(ch + u) * stride] : 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (ch + u < ch1) s += v[u];
    }
  }
  __shared__ float red[kBlock];
  red[tid()] = s;
  __syncthreads();
  if (gq == 0 && on) {
    float tot = red[el];
    for (int g = 1; g < ng; ++g) tot += red[g * ne + el];
    out[e] = tot;
    ql[e] = tot;
  }
}

// ---------------------------------------------------------------------------------------
// Decompress, general: M_hat = A B^T / p over a tile of rows.  Odd step: A = P_agg (factor
// buffer), B = Qh; even step: A = Ph, B = Q_agg.  B is staged in LDS column-major in chunks.
// Factor tiles keep the aggregated factor as the next step's reused factor and build its W.
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
    const float* src = src_of(a, d.bucket) + (odd ? d.fac_off_p : d.fac_off_q);
    float* dst = a.fac + (odd ? d.p_slot : d.q_slot);
    fact_tile<RK>(a, t, src, dst, odd ? d.n : d.m);
    return;
  }
  constexpr int CK = (8192 / RK) < 4096 ? (8192 / RK) : 4096;
  __shared__ __align__(16) float Bs[RK * CK];
  const float* agg = src_of(a, d.bucket);
  const float* A = odd ? agg + d.fac_off_p : a.fac + d.ph_slot;
  const float* B = odd ? a.fac + d.qh_slot : agg + d.fac_off_q;
  const int wave = tid() >> 6, lane = tid() & 63;
  const int64_t m = d.m;
  float* O = dst_of(a, d.bucket) + d.grad_off;
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
          float4 o = zero4();
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

// Decompress, r = 4: a row tile covers one block of 1024 columns (256 float4 groups, lane
// `lane` of wave w owns group 64 w + lane) of kReconRows rows taken with a stride (T_SROWS).  The
// planner orders the tiles so that workgroups launched together write adjacent whole rows: a
// small write footprint per workgroup with a dense band of rows across the running ones streams
// faster than long per-workgroup row blocks.  Each lane keeps the rank-4 rows of B for its
// columns in registers; stores are nontemporal tile-relative buffer stores: plain stores leave
// M_hat's lines dirty in the caches and the next step's kernels pay for writing them back.
// Factor tiles and vectors as in k_recon.
__global__ __launch_bounds__(kBlock) void k_recon4(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  const bool odd = a.parity != 0;
  if (t.kind == T_VEC) {
    vec_tile(a, t, false);
    return;
  }
  const MatDesc d = a.mats[t.idx];
  if (t.kind == T_FACT) {
    const float* src = src_of(a, d.bucket) + (odd ? d.fac_off_p : d.fac_off_q);
    float* dst = a.fac + (odd ? d.p_slot : d.q_slot);
    fact_tile<4>(a, t, src, dst, odd ? d.n : d.m);
    return;
  }
  if (t.kind == T_ROWS) {  // a narrow-row matrix's tile
    __shared__ float4 asn[kMaxTileRows];
    narrow_recon(a, t, d, asn);
    return;
  }
  if (t.kind == T_SMALL) {  // a small matrix, whole
    __shared__ float4 bsm[kSmallCols];
    small_recon(a, d, bsm);
    return;
  }
  const int cb = t.b & 15, stride = (t.b >> 4) & 0xfff, rows = t.b >> 16;
  const int m4 = d.m >> 2;
  const int g4 = (tid() >> 6) * 64 + (tid() & 63);  // float4 group within the block
  const int c4 = cb * 256 + g4;
  const bool ok = c4 < m4;
  const float* agg = src_of(a, d.bucket);
  const float4* A4 = reinterpret_cast<const float4*>(odd ? agg + d.fac_off_p : a.fac + d.ph_slot);
  const float4* B4 = reinterpret_cast<const float4*>(odd ? a.fac + d.qh_slot : agg + d.fac_off_q);
  __shared__ float4 as[kReconRows];  // the tile's rows of A, scaled by 1 / p
  if (tid() < rows) as[tid()] = scale4(A4[t.a + static_cast<int64_t>(tid()) * stride], a.inv_p);
  float4 b[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) b[c] = ok ? B4[4 * c4 + c] : zero4();
  __syncthreads();
  // the B rows are in registers before the stores, so no wait for them lands between them
  __builtin_amdgcn_s_waitcnt(0);
  const uint32_t row_bytes = static_cast<uint32_t>(d.m) * 4u;
  const uint32_t step_bytes = static_cast<uint32_t>(stride) * row_bytes;  // between tile rows
  const int cols = (d.m - cb * 1024) < 1024 ? (d.m - cb * 1024) : 1024;
  const Rsrc O = tile_rsrc(dst_of(a, d.bucket) + d.grad_off + static_cast<int64_t>(t.a) * d.m + cb * 1024,
                           static_cast<uint32_t>(rows - 1) * step_bytes + static_cast<uint32_t>(cols) * 4u);
  const uint32_t coff = ok ? static_cast<uint32_t>(g4) * 16u : kOut;
  // rows past the tile's count read unset LDS entries; their stores fall outside the resource
#pragma unroll
  for (int k = 0; k < kReconRows; ++k) {
    const float4 ar = as[k];
    const float4 o = make_float4(dot4(ar, b[0]), dot4(ar, b[1]), dot4(ar, b[2]), dot4(ar, b[3]));
    bst4_nt(O, static_cast<uint32_t>(k) * step_bytes + coff, o);
  }
}

__global__ __launch_bounds__(kBlock) void k_vec(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  vec_tile(a, t, true);
}


template <int RK>
hipError_t launch_rank(const Launch& l, const KArgs& args, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(l.ntiles)), block(kBlock);
  if constexpr (RK >= kBlockedRank) {  // only the kernels the r >= 8 launch lists use
    switch (l.kernel) {
      case K_APPLY: hipLaunchKernelGGL(k_apply<RK>, grid, block, 0, s, args); break;
      case K_EMAT: hipLaunchKernelGGL(k_emat<RK>, grid, block, 0, s, args); break;
      case K_FACT: hipLaunchKernelGGL(k_fact<RK>, grid, block, 0, s, args); break;
      case K_CHOL: hipLaunchKernelGGL(k_chol<RK>, grid, block, 0, s, args); break;
      case K_GSUM: hipLaunchKernelGGL(k_gsum<RK>, grid, block, 0, s, args); break;
      case K_QFIN: hipLaunchKernelGGL(k_qfin<RK>, grid, block, 0, s, args); break;
      case K_VEC: hipLaunchKernelGGL(k_vec, grid, block, 0, s, args); break;
      case K_DRAW: hipLaunchKernelGGL(k_draw<RK>, grid, block, 0, s, args); break;
      case K_IMAGE: hipLaunchKernelGGL(k_image<RK>, grid, block, 0, s, args); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  } else {
    switch (l.kernel) {
      case K_APPLY: hipLaunchKernelGGL(k_apply<RK>, grid, block, 0, s, args); break;
      case K_PROW: hipLaunchKernelGGL(k_prow<RK>, grid, block, 0, s, args); break;
      case K_EUPD: hipLaunchKernelGGL(k_eupd<RK>, grid, block, 0, s, args); break;
      case K_EMAT: hipLaunchKernelGGL(k_emat<RK>, grid, block, 0, s, args); break;
      case K_FACT: hipLaunchKernelGGL(k_fact<RK>, grid, block, 0, s, args); break;
      case K_CHOL: hipLaunchKernelGGL(k_chol<RK>, grid, block, 0, s, args); break;
      case K_QFIN: hipLaunchKernelGGL(k_qfin<RK>, grid, block, 0, s, args); break;
      case K_QSTEP:
        if (l.variant == (4 | kQFused)) {
          if constexpr (RK == 4) {
            hipLaunchKernelGGL((k_qstep<4, 4, true>), grid, block, 0, s, args);
          } else {
            return hipErrorInvalidValue;
          }
        } else if (l.variant == 4) {
          if constexpr (RK <= 8) {
            hipLaunchKernelGGL((k_qstep<RK, 4, false>), grid, block, 0, s, args);
          } else {
            return hipErrorInvalidValue;
          }
        } else if (l.variant == 1) {
          hipLaunchKernelGGL((k_qstep<RK, 1, false>), grid, block, 0, s, args);
        } else {
          return hipErrorInvalidValue;
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
            case 1 | kThreeWaves:
              hipLaunchKernelGGL((k_pfused<1, 3>), grid, dim3(3 * kWave), 0, s, args);
              break;
            case 2 | kEightWaves:
              hipLaunchKernelGGL((k_pfused<2, 8>), grid, dim3(8 * kWave), 0, s, args);
              break;
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
      case K_RECON4:
        if constexpr (RK == 4) {
          hipLaunchKernelGGL(k_recon4, grid, block, 0, s, args);
          break;
        } else {
          return hipErrorInvalidValue;
        }
      case K_VEC: hipLaunchKernelGGL(k_vec, grid, block, 0, s, args); break;
      case K_DRAW: hipLaunchKernelGGL(k_draw<RK>, grid, block, 0, s, args); break;
      case K_IMAGE: hipLaunchKernelGGL(k_image<RK>, grid, block, 0, s, args); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
}

}  // namespace

hipError_t launch(const Launch& l, int32_t rank, const KArgs& args, hipStream_t s) {
  if (l.ntiles <= 0) return hipSuccess;
  if (l.kernel == K_WPSTEP || l.kernel == K_WQSTEP || l.kernel == K_WRECON || l.kernel == K_WFACT)
    return launch_wide(l, rank, args, s);
  switch (rank) {
    case 1: return launch_rank<1>(l, args, s);
    case 2: return launch_rank<2>(l, args, s);
    case 4: return launch_rank<4>(l, args, s);
    case 8: return launch_rank<8>(l, args, s);
    case 16: return launch_rank<16>(l, args, s);
    case 32: return launch_rank<32>(l, args, s);
    case 64: return launch_rank<64>(l, args, s);
    case 128: return launch_rank<128>(l, args, s);
    case 256: return launch_rank<256>(l, args, s);
    default: return hipErrorInvalidValue;
  }
}

// Q-step partials of acp_compress_noalloc: a file-scope device array, one copy on every GPU the
// library runs on, kept until the process ends.  In host code its name is only a symbol, not a
// device address: scratch_address() looks up the current device's copy once with
// hipGetSymbolAddress and keeps that address per device; every launch takes the address.
static __device__ __align__(256) float scratch[kScratchBytes / 4];

hipError_t scratch_address(int device, float** out) {
  static std::mutex mu;
  static std::vector<float*> addr;  // per device; null until looked up
  std::lock_guard<std::mutex> lock(mu);
  if (device < 0) return hipErrorInvalidDevice;
  if (addr.size() <= static_cast<size_t>(device)) addr.resize(static_cast<size_t>(device) + 1, nullptr);
  if (!addr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[device] = static_cast<float*>(p);
  }
  *out = addr[device];
  return hipSuccess;
}

}  // namespace acp
