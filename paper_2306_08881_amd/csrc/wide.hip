// gfx950 MFMA kernels of the ACP-SGD compressor for ranks 8 to 256 (arXiv 2306.08881,
// Algorithm 2).  At these ranks a step costs 2r multiply-adds per gradient element against
// 12 bytes of HBM traffic, more than the fp32 vector units sustain at full bandwidth, so the
// rank-r contractions run on v_mfma_f32_32x32x2f32.
//
// Both compress steps apply the error-feedback residual of the previous step in deferred
// form and write M' back, so neither waits for its own reduction before writing:
//   P-step:  X = M + E_arena (- Ph Ql^T when the arena holds F), X written to the arena,
//            P_loc = X Qh;  afterwards E = X - P_loc Qh^T is implied.
//   Q-step:  F = M + E_arena (- Pl Qh^T when the arena holds X), F written to the arena,
//            Q_loc = F^T Ph; afterwards E = F - Ph Q_loc^T is implied.
// Each is one rank-r correction and one rank-r product per element.  From rank 64 the waves of
// a workgroup split the rank in the compress kernels (k_spstep, k_sqstep), at rank 256 in the
// decompress kernel too (k_srecon); the one-wave decompress keeps r / 32 output blocks per wave.
//
// MFMA layout (one wave): D (32 x 32) += A (32 x 2) B (2 x 32).  Lane l supplies
// A[l % 32][l / 32] and B[l / 32][l % 32]; register v of lane l holds D[drow(v, l / 32)][l % 32].
// The K index of a step may map to any pair of rank (or row, column) indices as long as A and
// B use the same pair; the kernels use rank (r / 2) h + s on half h at step s, and the row or
// column drow(v, h) at step v, which lets the output of one MFMA feed the next directly.
#include "device.hpp"

#include <type_traits>

namespace acp {

namespace {

typedef float v16f __attribute__((ext_vector_type(16)));

__device__ inline v16f mfma(float a, float b, const v16f& c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}
__device__ inline int drow(int v, int h) { return 8 * (v >> 2) + 4 * h + (v & 3); }
__device__ inline v16f zero16() {
  v16f z;
#pragma unroll
  for (int v = 0; v < 16; ++v) z[v] = 0.f;
  return z;
}
__device__ inline uint32_t u32(int64_t x) { return static_cast<uint32_t>(x); }

// KH consecutive floats of a factor row starting at byte offset off (kOut: zeros); with
// vec, four at a time (the resource base and off are 16-byte aligned).
template <int KH>
__device__ inline void load_run(Rsrc r, uint32_t off, bool vec, float* out) {
  if (vec) {
#pragma unroll
    for (int i = 0; i < KH / 4; ++i) {
      const float4 f = bld4(r, off == kOut ? kOut : off + 16u * i);
      out[4 * i + 0] = f.x;
      out[4 * i + 1] = f.y;
      out[4 * i + 2] = f.z;
      out[4 * i + 3] = f.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < KH; ++i) out[i] = bld1(r, off == kOut ? kOut : off + 4u * i);
  }
}
__device__ inline bool aligned16(const float* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// P-step over a tile of at most 32 rows and all m columns on four waves: wave w walks the
// 32-column blocks w, w + 4, ... in step with the others, so that the workgroup reads 512
// contiguous bytes of each of its rows at a time.  Per step of 128 columns, wave w loads M and E
// for rows 8 w ... 8 w + 7 as 16-byte vectors (lane l: row 8 w + 2 i + l / 32, columns
// 4 (l % 32) ... + 3; one instruction reads 512 contiguous bytes of two rows), puts M + E in a
// 32 x 128 LDS tile, and after a barrier takes its own block back with lane l holding column
// c0 + l % 32 of rows drow(v, l / 32).  It applies the correction (F form) as an MFMA with D
// indexed (row, column).  The product P += X Qh reduces over columns, so it needs the row on the
// lane: X goes through the wave's padded 32 x 33 LDS tile (two of them, alternating) and comes
// back with lane l holding row l % 32 and columns drow(v, l / 32), the A operand; the
// accumulator lane l holds the wave's share of P[r0 + drow(v, l / 32)][l % 32].  After the
// barrier that publishes those tiles, every wave also reads its rows of X in the load layout
// from the four waves' tiles and stores them as 16-byte vectors.  The four shares of P are added
// in wave order through LDS at the end.  The next step's M and E are requested before the
// current block's MFMAs, its factor rows after them.
template <int RK>
__global__ __launch_bounds__(kWideBlock * kWidePWaves, 2) void k_wpstep(KArgs a) {
  constexpr int KH = RK / 2;
  constexpr int NR = RK > 32 ? RK / 32 : 1;  // 32-rank blocks of P (one MFMA block each)
  constexpr int LD = 33;  // padded LDS row: the transposed reads hit 32 different banks
  constexpr int CS = 32 * kWidePWaves;  // columns per step of the workgroup
  const Tile t = a.tiles[blockIdx.x];
  if (t.kind == T_VEC) {  // a raw vector packed into the factor buffer
    vec_tile(a, t, true);
    return;
  }
  const MatDesc d = a.mats[t.idx];
  const int wave = __builtin_amdgcn_readfirstlane(tid() >> 6);
  const int lane = tid() & 63, h = lane >> 5, li = lane & 31;
  const int64_t m = d.m, r0 = t.a;
  const int rows = t.b;
  const bool fform = deferred_of(a, d.bucket);
  const uint32_t row_bytes = u32(m) * 4u;
  const uint32_t ext = u32(rows) * row_bytes;
  const Rsrc G = tile_rsrc(src_of(a, d.bucket) + d.grad_off + r0 * m, ext);
  const Rsrc E = tile_rsrc(a.e + d.e_off + r0 * m, a.ef ? ext : 0u);
  const Rsrc Phr = tile_rsrc(a.fac + d.ph_slot + r0 * RK, fform ? u32(rows) * RK * 4u : 0u);
  const Rsrc Qlr = tile_rsrc(a.fac + d.ql_slot, fform ? u32(m) * RK * 4u : 0u);
  const Rsrc Qhr = tile_rsrc(a.fac + d.qh_slot, u32(m) * RK * 4u);
  const bool ph4 = aligned16(a.fac + d.ph_slot), ql4 = aligned16(a.fac + d.ql_slot);
  static_assert(RK < kSplitRank, "from kSplitRank on the rank-split kernel takes the P-step");
  float pa[KH];  // correction A operand: -Ph[r0 + l % 32][KH h + s]
  load_run<KH>(Phr, u32(li * RK + KH * h) * 4u, ph4, pa);
#pragma unroll
  for (int s = 0; s < KH; ++s) pa[s] = -pa[s];

  // M and E of the step from column cs: the lane's four rows 8 w + 2 i + h, columns cs + 4 li ...
  // (past m: zeros); as 16-byte vectors when rows and tile starts are 16-byte aligned, else
  // float by float in the same layout
  const bool vec = (m & 3) == 0 && aligned16(src_of(a, d.bucket) + d.grad_off + r0 * m) &&
                   aligned16(a.e + d.e_off + r0 * m);
  const int vr = 8 * wave + h, vc = 4 * li;
  auto load_block = [&](int64_t cs, float4* g, float4* e) {
    const int64_t col = cs + vc;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t o = u32(vr + 2 * i) * row_bytes + u32(col) * 4u;
      if (vec) {
        g[i] = bld4_nt(G, col < m ? o : kOut);
        e[i] = bld4_nt(E, col < m ? o : kOut);
      } else {
        g[i] = make_float4(bld1_nt(G, col < m ? o : kOut), bld1_nt(G, col + 1 < m ? o + 4u : kOut),
                           bld1_nt(G, col + 2 < m ? o + 8u : kOut), bld1_nt(G, col + 3 < m ? o + 12u : kOut));
        e[i] = make_float4(bld1_nt(E, col < m ? o : kOut), bld1_nt(E, col + 1 < m ? o + 4u : kOut),
                           bld1_nt(E, col + 2 < m ? o + 8u : kOut), bld1_nt(E, col + 3 < m ? o + 12u : kOut));
      }
    }
  };
  // the block's factor operands: Ql rows (correction B) and Qh rows (product B, rank block kb)
  auto load_ops = [&](int64_t c0, float* qa, float (*qb)[16]) {
    const int64_t qcol = c0 + li;
    if (fform) load_run<KH>(Qlr, qcol < m ? u32(qcol * RK + KH * h) * 4u : kOut, ql4, qa);
#pragma unroll
    for (int kb = 0; kb < NR; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t col = c0 + drow(v, h);
        const int rank = kb * 32 + li;
        qb[kb][v] = bld1(Qhr, (col < m && rank < RK) ? u32(col * RK + rank) * 4u : kOut);
      }
  };
  // the waves' transposing tiles, two each; a wave's pair starts one float past the previous
  // wave's, so that the row reads of the X stores (four waves' tiles at once) spread over the banks
  constexpr int XW = 2 * 32 * LD + 1;
  __shared__ float xt[kWidePWaves * XW];
  auto xtile = [&](int w, int b) { return xt + w * XW + b * 32 * LD; };
  constexpr int SP = 32 * kWidePWaves + 4;  // staging tile row pitch (floats, 16-byte aligned rows)
  __shared__ __attribute__((aligned(16))) float st[32 * SP];
  float4 g[4], e[4];
  float qa[KH], qb[NR][16];
  load_block(0, g, e);
  load_ops(32 * wave, qa, qb);

  v16f p[NR];
#pragma unroll
  for (int kb = 0; kb < NR; ++kb) p[kb] = zero16();
  int buf = 0;
  // every wave takes the same number of steps (blocks past m: zero loads, dropped stores)
  for (int64_t cs = 0; cs < m; cs += CS, buf ^= 1) {
    const int64_t c0 = cs + 32 * wave;
    // M + E to the staging tile (the previous step's readers have passed its second barrier)
#pragma unroll
    for (int i = 0; i < 4; ++i) *reinterpret_cast<float4*>(st + (vr + 2 * i) * SP + vc) = g[i] + e[i];
    load_block(cs + CS, g, e);  // next step (past m: zeros, no traffic)
    __syncthreads();
    v16f x;
#pragma unroll
    for (int v = 0; v < 16; ++v) x[v] = st[drow(v, h) * SP + 32 * wave + li];
    if (fform) {  // X -= Ph Ql^T: A = -Ph (row, rank), B = Ql^T (rank, column)
#pragma unroll
      for (int s = 0; s < KH; ++s) x = mfma(pa[s], qa[s], x);
    }
    float* tl = xtile(wave, buf);
#pragma unroll
    for (int v = 0; v < 16; ++v) tl[drow(v, h) * LD + li] = x[v];
    __syncthreads();
    // X to the arena in the load layout: the lane's rows 8 w + 2 i + h, columns cs + 4 li ...,
    // from the transposing tile of the wave that formed them (as 16-byte vectors when aligned)
    {
      const float* xs = xtile(li >> 3, buf) + (vc & 31);
      const int64_t col = cs + vc;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = vr + 2 * i;
        const float4 xv = make_float4(xs[row * LD], xs[row * LD + 1], xs[row * LD + 2], xs[row * LD + 3]);
        const uint32_t o = u32(row) * row_bytes + u32(col) * 4u;
        if (vec) {
          bst4_nt(E, col < m ? o : kOut, xv);
        } else {
          bst1_nt(E, col < m ? o : kOut, xv.x);
          bst1_nt(E, col + 1 < m ? o + 4u : kOut, xv.y);
          bst1_nt(E, col + 2 < m ? o + 8u : kOut, xv.z);
          bst1_nt(E, col + 3 < m ? o + 12u : kOut, xv.w);
        }
      }
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) {  // P += X Qh: A = X (row, column), B = Qh (column, rank)
      const float xa = tl[li * LD + drow(v, h)];
#pragma unroll
      for (int kb = 0; kb < NR; ++kb) p[kb] = mfma(xa, qb[kb][v], p[kb]);
    }
    load_ops(c0 + CS, qa, qb);
  }

  // the waves' shares of P, added in wave order: entry (v, lane) of rank block kb
  float* red = xt;  // kWidePWaves x 1024 floats per rank block (the transposing tiles are free)
  float* P = dst_of(a, d.bucket) + d.fac_off_p;
  float* Pl = a.fac + d.pl_slot;
#pragma unroll
  for (int kb = 0; kb < NR; ++kb) {
    __syncthreads();  // the last products have read the tiles (and the previous block's sums)
#pragma unroll
    for (int v = 0; v < 16; ++v) red[wave * 1024 + v * 64 + lane] = p[kb][v];
    __syncthreads();
    for (int en = tid(); en < 1024; en += kWideBlock * kWidePWaves) {
      float sum = red[en];
#pragma unroll
      for (int q = 1; q < kWidePWaves; ++q) sum += red[q * 1024 + en];
      const int v = en >> 6, ln = en & 63;
      const int row = drow(v, ln >> 5), rank = kb * 32 + (ln & 31);
      if (rank < RK && row < rows) {
        P[(r0 + row) * RK + rank] = sum;
        Pl[(r0 + row) * RK + rank] = sum;
      }
    }
  }
}

// Q-step over a tile (row chunk t.a of q_rows rows, column blocks 4 t.b ... 4 t.b + 3 of 32
// columns), four waves per workgroup: wave w takes column block 4 t.b + w (columns c0 ...
// c0 + 31) and the waves walk the chunk's 32-row blocks in step, so that the workgroup reads 512
// contiguous bytes of each row at a time.  Per 32-row block, wave w loads M and E for rows
// 8 w ... 8 w + 7 of the workgroup's 128 columns as 16-byte vectors (as the P-step does), puts
// M + E in a 32 x 128 LDS tile and after a barrier takes its own block back with lane l holding
// column c0 + l % 32 of rows drow(v, l / 32).  The block's Pl and Ph rows are loaded once for
// the workgroup into a factor tile beside it.  The correction (X form) is an MFMA with D indexed
// (row, column); F then is the A operand of Q += F^T Ph with the rows as K, and goes back into
// the wave's block of the tile, from which every wave stores its rows of F as 16-byte vectors
// after the block's last barrier.  Lane l's partial Q of column c0 + drow(v, l / 32), rank
// l % 32, goes to the chunk's partial block for K_QFIN.
template <int RK>
__global__ __launch_bounds__(kWideBlock * kWideQWaves, 2) void k_wqstep(KArgs a) {
  constexpr int KH = RK / 2;
  constexpr int NR = RK > 32 ? RK / 32 : 1;  // 32-rank blocks of Q (one MFMA block each)
  const Tile t = a.tiles[blockIdx.x];
  const MatDesc d = a.mats[t.idx];
  const int wave = __builtin_amdgcn_readfirstlane(tid() >> 6);
  const int lane = tid() & 63, h = lane >> 5, li = lane & 31;
  const int64_t n = d.n, m = d.m;
  const int64_t r0 = static_cast<int64_t>(t.a) * d.q_rows;
  const int rows = static_cast<int>((r0 + d.q_rows < n) ? d.q_rows : n - r0);
  const int64_t c0 = (static_cast<int64_t>(t.b) * kWideQWaves + wave) * d.q_cb;
  // valid columns of the wave's block: none for a block past m (its wave loads zeros, stores
  // nothing and keeps the others' barriers)
  const int64_t w = (m - c0) < 32 ? ((m - c0) > 0 ? (m - c0) : 0) : 32;
  const bool xform = deferred_p_of(a, d.bucket);
  const uint32_t row_bytes = u32(m) * 4u;
  // the workgroup's columns ct ... ct + wt - 1
  const int64_t ct = static_cast<int64_t>(t.b) * kWideQWaves * d.q_cb;
  const int64_t wt = (m - ct) < 32 * kWideQWaves ? m - ct : 32 * kWideQWaves;
  const uint32_t extw = u32(rows - 1) * row_bytes + u32(wt) * 4u;
  const float* gbase = src_of(a, d.bucket) + d.grad_off + r0 * m + ct;
  const float* ebase = a.e + d.e_off + r0 * m + ct;
  const Rsrc Gw = tile_rsrc(gbase, extw);
  const Rsrc Ew = tile_rsrc(ebase, a.ef ? extw : 0u);
  const bool vec = (m & 3) == 0 && aligned16(gbase) && aligned16(ebase);
  const Rsrc Qhr = tile_rsrc(a.fac + d.qh_slot + c0 * RK, xform ? u32(w) * RK * 4u : 0u);
  const Rsrc Plr = tile_rsrc(a.fac + d.pl_slot + r0 * RK, xform ? u32(rows) * RK * 4u : 0u);
  const Rsrc Phr = tile_rsrc(a.fac + d.ph_slot + r0 * RK, u32(rows) * RK * 4u);
  static_assert(RK < kSplitRank, "from kSplitRank on the rank-split kernel takes the Q-step");
  float qv[KH];  // correction B operand: Qh[c0 + l % 32][KH h + s]
#pragma unroll
  for (int s = 0; s < KH; ++s) qv[s] = bld1(Qhr, u32(li * RK + KH * h + s) * 4u);

  // M and E of the 32-row block from row rb: the lane's rows rb + 8 w + 2 i + h, columns
  // 4 li ... 4 li + 3 of the workgroup's (past wt or the chunk: zeros); 16-byte vectors when the
  // rows and the first column are 16-byte aligned, else float by float in the same layout
  const int vr = 8 * wave + h, vc = 4 * li;
  auto load_block = [&](int rb, float4* g, float4* e) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t o = u32(rb + vr + 2 * i) * row_bytes + u32(vc) * 4u;
      if (vec) {
        g[i] = bld4_nt(Gw, vc < wt ? o : kOut);
        e[i] = bld4_nt(Ew, vc < wt ? o : kOut);
      } else {
        g[i] = make_float4(bld1_nt(Gw, vc < wt ? o : kOut), bld1_nt(Gw, vc + 1 < wt ? o + 4u : kOut),
                           bld1_nt(Gw, vc + 2 < wt ? o + 8u : kOut), bld1_nt(Gw, vc + 3 < wt ? o + 12u : kOut));
        e[i] = make_float4(bld1_nt(Ew, vc < wt ? o : kOut), bld1_nt(Ew, vc + 1 < wt ? o + 4u : kOut),
                           bld1_nt(Ew, vc + 2 < wt ? o + 8u : kOut), bld1_nt(Ew, vc + 3 < wt ? o + 12u : kOut));
      }
    }
  };
  // the block's factor rows, Pl (correction A) and Ph (product B): 32 x RK contiguous floats each
  // (factor slots are 256-byte aligned), loaded once for the workgroup, one 16-byte word per
  // thread, into a factor tile beside the staging tile, from which every wave takes its operands
  static_assert(NR == 1, "one 32-rank block below kSplitRank");
  constexpr int FP = RK + 4;        // factor tile row pitch (floats, 16-byte aligned rows)
  constexpr int FV = 32 * RK / 4;   // 16-byte words per block and factor
  const bool fw = tid() < FV;       // the thread has a word of the block
  const int frow = tid() * 4 / RK, fcol = tid() * 4 % RK;
  auto load_fac = [&](int rb, float4& l, float4& p) {
    const uint32_t o = u32(rb * RK + tid() * 4) * 4u;
    l = bld4(Plr, fw ? o : kOut);  // zeros past the chunk, and without the X form
    p = bld4(Phr, fw ? o : kOut);
  };
  // two staging tiles in turn: block k's F goes back into tile k % 2 and is stored from there
  // after the block's last barrier, while block k + 1 fills the other
  constexpr int SP = 32 * kWideQWaves + 4;  // staging tile row pitch (floats, 16-byte aligned rows)
  __shared__ __attribute__((aligned(16))) float st[2][32 * SP];
  __shared__ __attribute__((aligned(16))) float ft[2][2][32 * FP];  // [tile][Pl, Ph]
  float4 g[4], e[4], fl, fh;
  load_block(0, g, e);
  load_fac(0, fl, fh);
  v16f q[NR];
#pragma unroll
  for (int kb = 0; kb < NR; ++kb) q[kb] = zero16();
  int buf = 0;
  for (int rb = 0; rb < rows; rb += 32, buf ^= 1) {
    float* sb = st[buf];
    float* fpl = ft[buf][0];
    float* fph = ft[buf][1];
    // M + E and the factor rows to the tiles (their readers of two blocks ago have passed the
    // last barrier)
#pragma unroll
    for (int i = 0; i < 4; ++i) *reinterpret_cast<float4*>(sb + (vr + 2 * i) * SP + vc) = g[i] + e[i];
    if (fw) {
      *reinterpret_cast<float4*>(fpl + frow * FP + fcol) = fl;
      *reinterpret_cast<float4*>(fph + frow * FP + fcol) = fh;
    }
    load_block(rb + 32, g, e);  // next block (past the chunk: zeros, no traffic)
    load_fac(rb + 32, fl, fh);
    __syncthreads();
    v16f x;
#pragma unroll
    for (int v = 0; v < 16; ++v) x[v] = sb[drow(v, h) * SP + 32 * wave + li];
    if (xform) {  // F -= Pl Qh^T: A = -Pl (row, rank), B = Qh^T (rank, column)
      float pa[KH];  // Pl[rb + l % 32][KH h + s]
#pragma unroll
      for (int s = 0; s < KH; ++s) pa[s] = fpl[li * FP + KH * h + s];
#pragma unroll
      for (int s = 0; s < KH; ++s) x = mfma(-pa[s], qv[s], x);
    }
    // F back into the wave's own block of the tile (only this wave has read it)
#pragma unroll
    for (int v = 0; v < 16; ++v) sb[drow(v, h) * SP + 32 * wave + li] = x[v];
    {  // Q += F^T Ph: A = F^T, B = Ph (lane l: rank l % 32 of rows drow(v, l / 32); zero past r)
      const int rk = li < RK ? li : RK - 1;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float pb = fph[drow(v, h) * FP + rk];
        q[0] = mfma(x[v], li < RK ? pb : 0.f, q[0]);
      }
    }
    __syncthreads();  // the waves stay on the same rows; every block's F is in the tile
    // F to the arena in the load layout, as 16-byte vectors when aligned
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float4 f = *reinterpret_cast<const float4*>(sb + (vr + 2 * i) * SP + vc);
      const uint32_t o = u32(rb + vr + 2 * i) * row_bytes + u32(vc) * 4u;
      if (vec) {
        bst4_nt(Ew, vc < wt ? o : kOut, f);
      } else {
        bst1_nt(Ew, vc < wt ? o : kOut, f.x);
        bst1_nt(Ew, vc + 1 < wt ? o + 4u : kOut, f.y);
        bst1_nt(Ew, vc + 2 < wt ? o + 8u : kOut, f.z);
        bst1_nt(Ew, vc + 3 < wt ? o + 12u : kOut, f.w);
      }
    }
  }
  if (w == 0) return;  // a block past m has no partials
  const int64_t ncb = (m + d.q_cb - 1) / d.q_cb;
  const int64_t stride = ncb * d.q_cb * RK;  // one row chunk of partials
  float* part = a.qpart + d.qpart + static_cast<int64_t>(t.a) * stride + c0 * RK;
#pragma unroll
  for (int kb = 0; kb < NR; ++kb) {
    const int rank = kb * 32 + li;
    if (rank < RK)
#pragma unroll
      for (int v = 0; v < 16; ++v) part[drow(v, h) * RK + rank] = q[kb][v];
  }
}

// Decompress from rank 64 (the four-wave kernel below takes the lower ranks): M_hat = A B^T / p
// over a tile (32-row block t.a, 1024-column group t.b), one wave per workgroup walking the
// group's 32-column blocks in bursts.  Odd step: A = P_agg (factor buffer), B = Qh; even step:
// A = Ph, B = Q_agg.  A burst of BURST blocks is computed into one accumulator block each, then
// stored row pair by row pair: lane l stores column c0 + l % 32 of rows drow(v, l / 32) for each
// block of the burst in turn.  Stores are nontemporal (plain stores leave M_hat's lines dirty in
// the caches, and the next step's kernels pay for writing them back).  Each block's B rows are
// requested one block ahead of its MFMAs.
template <int RK>
__global__ __launch_bounds__(kWideBlock) void k_wrecon(KArgs a) {
  constexpr int KH = RK / 2;
  constexpr int NB = kWideRCols / 32;                          // column blocks per tile
  constexpr int BURST = RK <= 64 ? 2 : 1;  // blocks per burst (accumulators)
  static_assert(NB % (2 * BURST) == 0, "pairs of bursts tile the column group");
  const Tile t = a.tiles[blockIdx.x];
  const bool odd = a.parity != 0;
  const MatDesc d = a.mats[t.idx];
  const int lane = tid(), h = lane >> 5, li = lane & 31;
  const int64_t n = d.n, m = d.m;
  const int64_t r0 = static_cast<int64_t>(t.a) * 32;
  const int rows = static_cast<int>((r0 + 32 < n) ? 32 : n - r0);
  const float* agg = src_of(a, d.bucket);
  const float* A = odd ? agg + d.fac_off_p : a.fac + d.ph_slot;
  const float* B = odd ? a.fac + d.qh_slot : agg + d.fac_off_q;
  const Rsrc Ar = tile_rsrc(A + r0 * RK, u32(rows) * RK * 4u);
  const Rsrc Br = tile_rsrc(B, u32(m) * RK * 4u);
  const bool a4 = aligned16(A), b4 = aligned16(B);
  float av[KH];  // A operand: A[r0 + l % 32][KH h + s] / p
  load_run<KH>(Ar, u32(li * RK + KH * h) * 4u, a4, av);
#pragma unroll
  for (int s = 0; s < KH; ++s) av[s] *= a.inv_p;
  float* O = dst_of(a, d.bucket) + d.grad_off + r0 * m;
  const uint32_t row_bytes = u32(m) * 4u;
  // one resource over the tile's rows: rows past `rows` fall outside it; columns past m are masked
  const Rsrc Or = tile_rsrc(O, u32(rows) * row_bytes);
  const uint32_t lane_row = u32(4 * h) * row_bytes;  // drow(v, h) = 8 (v / 4) + v % 4 + 4 h
  auto bcol = [&](int j) { return static_cast<int64_t>(t.b) * kWideRCols + j * 32; };
  auto boff = [&](int j) { return bcol(j) + li < m ? u32((bcol(j) + li) * RK + KH * h) * 4u : kOut; };
  float bv[2][KH];  // B operand: B[c0 + l % 32][KH h + s] of block j in bv[j % 2], and the next
  load_run<KH>(Br, boff(0), b4, bv[0]);
  // one burst from block j0, whose parity P is a compile-time constant (register indices are)
  auto burst = [&](int j0, auto parity) {
    constexpr int P = decltype(parity)::value;
    // the products: block j0 + jb into o[jb], the next block's B rows requested first
    v16f o[BURST];
#pragma unroll
    for (int jb = 0; jb < BURST; ++jb) {
      if (j0 + jb + 1 < NB) load_run<KH>(Br, boff(j0 + jb + 1), b4, bv[(P + jb + 1) & 1]);
      o[jb] = zero16();
#pragma unroll
      for (int s = 0; s < KH; ++s) o[jb] = mfma(av[s], bv[(P + jb) & 1][s], o[jb]);
    }
    // the stores: the lane's offset per block (kOut past m), to which each row adds a
    // wave-uniform part; the empty asm keeps the compiler from carrying a running offset per row
    const int64_t cb = bcol(j0);
    const int wb = static_cast<int>((m - cb) < BURST * 32 ? (m - cb) : BURST * 32);
    uint32_t base = lane_row + u32(cb + li) * 4u;
    asm volatile("" : "+v"(base));
    uint32_t bo[BURST];
#pragma unroll
    for (int jb = 0; jb < BURST; ++jb) bo[jb] = jb * 32 + li < wb ? base + u32(jb * 128) : kOut;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const uint32_t roff = u32(8 * (v >> 2) + (v & 3)) * row_bytes;
#pragma unroll
      for (int jb = 0; jb < BURST; ++jb) bst1_nt(Or, bo[jb] + roff, o[jb][v]);
    }
  };
  // two bursts per iteration: the first starts on an even block, the second on block j0 + BURST
  for (int j0 = 0; j0 < NB; j0 += 2 * BURST) {
    if (bcol(j0) >= m) break;
    burst(j0, std::integral_constant<int, 0>{});
    if (bcol(j0 + BURST) >= m) break;
    burst(j0 + BURST, std::integral_constant<int, BURST & 1>{});
  }
}

// Decompress up to rank 32 with four waves per tile (32-row block t.a, 1024-column group t.b):
// at step k the waves compute the 32 x 32 blocks 4k ... 4k + 3 (wave w block 4k + w), as the
// one-wave kernel does, and put them in an LDS tile of 32 rows x 128 columns; then all 256
// threads store that tile with 16-byte nontemporal stores, thread t taking the four columns
// 4 (t % 32) ... of rows t / 32 + 8 i, so one store instruction writes 512 contiguous bytes of
// each of two rows (the one-wave kernel's stores write 128 bytes of a row at a time).  Two LDS
// tiles alternate, one barrier per step.  Rows past the tile fall outside the output resource;
// columns past m are masked per float (16-byte stores need m and the tile start 16-byte aligned,
// otherwise the same layout is stored float by float).
template <int RK>
__global__ __launch_bounds__(kBlock) void k_wrecon4w(KArgs a) {
  constexpr int KH = RK / 2;
  constexpr int LP = 132;  // LDS row pitch (floats): rows stay 16-byte aligned for the reads
  const Tile t = a.tiles[blockIdx.x];
  const bool odd = a.parity != 0;
  const MatDesc d = a.mats[t.idx];
  const int wave = __builtin_amdgcn_readfirstlane(tid() >> 6);
  const int lane = tid() & 63, h = lane >> 5, li = lane & 31;
  const int64_t n = d.n, m = d.m;
  const int64_t r0 = static_cast<int64_t>(t.a) * 32;
  const int rows = static_cast<int>((r0 + 32 < n) ? 32 : n - r0);
  const float* agg = src_of(a, d.bucket);
  const float* A = odd ? agg + d.fac_off_p : a.fac + d.ph_slot;
  const float* B = odd ? a.fac + d.qh_slot : agg + d.fac_off_q;
  const Rsrc Ar = tile_rsrc(A + r0 * RK, u32(rows) * RK * 4u);
  const Rsrc Br = tile_rsrc(B, u32(m) * RK * 4u);
  const bool a4 = aligned16(A), b4 = aligned16(B);
  float av[KH];  // A operand: A[r0 + l % 32][KH h + s] / p
  load_run<KH>(Ar, u32(li * RK + KH * h) * 4u, a4, av);
#pragma unroll
  for (int s = 0; s < KH; ++s) av[s] *= a.inv_p;
  float* O = dst_of(a, d.bucket) + d.grad_off + r0 * m;
  const uint32_t row_bytes = u32(m) * 4u;
  const Rsrc Or = tile_rsrc(O, u32(rows) * row_bytes);
  const bool vec = (m & 3) == 0 && aligned16(O);
  const int64_t c0 = static_cast<int64_t>(t.b) * kWideRCols;
  constexpr int NS = kWideRCols / 128;  // steps of four blocks
  auto bcol = [&](int k) { return c0 + k * 128 + wave * 32; };  // the wave's block at step k
  auto boff = [&](int k) { return bcol(k) + li < m ? u32((bcol(k) + li) * RK + KH * h) * 4u : kOut; };
  __shared__ __attribute__((aligned(16))) float tile[2][32 * LP];
  float bv[2][KH];
  load_run<KH>(Br, boff(0), b4, bv[0]);
  const int sc = tid() & 31, sr = tid() >> 5;  // store side: float4 column sc of rows sr + 8 i
  for (int k = 0; k < NS; ++k) {
    const int64_t cs = c0 + k * 128;  // the step's first column
    if (cs >= m) break;
    if (k + 1 < NS) load_run<KH>(Br, boff(k + 1), b4, bv[(k + 1) & 1]);
    v16f o = zero16();
#pragma unroll
    for (int s = 0; s < KH; ++s) o = mfma(av[s], bv[k & 1][s], o);
    float* tl = tile[k & 1];
#pragma unroll
    for (int v = 0; v < 16; ++v) tl[drow(v, h) * LP + wave * 32 + li] = o[v];
    __syncthreads();
    const int64_t col = cs + 4 * sc;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = sr + 8 * i;
      const float4 q = *reinterpret_cast<const float4*>(tl + r * LP + 4 * sc);
      const uint32_t off = u32(r) * row_bytes + u32(col) * 4u;
      if (vec) {
        bst4_nt(Or, col < m ? off : kOut, q);
      } else {
        bst1_nt(Or, col < m ? off : kOut, q.x);
        bst1_nt(Or, col + 1 < m ? off + 4u : kOut, q.y);
        bst1_nt(Or, col + 2 < m ? off + 8u : kOut, q.z);
        bst1_nt(Or, col + 3 < m ? off + 12u : kOut, q.w);
      }
    }
  }
}

// ---------------------------------------------------------------------------------------
// From kSplitRank on one wave cannot hold the operands of every rank, so the SW waves of a
// workgroup (split_waves: 2 at rank 64, 4 from rank 128) split the rank: wave w takes ranks
// rk0 = w r / SW ... of each rank-r term (r / 2 SW K steps per lane half, r / 32 SW 32-rank
// output blocks), with the operand layout of the kernels above.  A correction (or a
// decompressed block) is a sum over all ranks, so each wave writes its partial 32 x 32 block to
// LDS and wave w adds the SW partials, in wave order, for its EPW = 16 / SW entries
// v = EPW w + j (j < EPW) of the MFMA layout, rows drow(v, l / 32) of the block.  Wave w also
// loads M and E for those entries only.  LDS buffers alternate between blocks, so one barrier
// per use suffices.
constexpr int split_waves(int r) { return r >= 128 ? 4 : 2; }

// P-step over a 32-row tile, the 32-column blocks in order: partial corrections -Ph Ql^T (F
// form) -> X = M + E + their sum for the wave's entries, stored to the arena and to the
// transposing tile -> P += X Qh over the wave's ranks.  The next block's M, E and factor rows are
// requested before the current block's MFMAs.
template <int RK>
__global__ __launch_bounds__(kWave * split_waves(RK), 2) void k_spstep(KArgs a) {
  constexpr int SW = split_waves(RK), EPW = 16 / SW, RS = RK / SW, KH = RS / 2, NR = RS / 32;
  static_assert(RS % 32 == 0 && EPW * SW == 16, "whole 32-rank blocks and entries per wave");
  constexpr int LD = 33;
  const Tile t = a.tiles[blockIdx.x];
  if (t.kind == T_VEC) {  // a raw vector packed into the factor buffer
    vec_tile(a, t, true);
    return;
  }
  const MatDesc d = a.mats[t.idx];
  const int wave = tid() >> 6, lane = tid() & 63, h = lane >> 5, li = lane & 31;
  const int rk0 = wave * RS;
  const int64_t m = d.m, r0 = t.a;
  const int rows = t.b;
  const bool fform = deferred_of(a, d.bucket);
  const uint32_t row_bytes = u32(m) * 4u;
  const uint32_t ext = u32(rows) * row_bytes;
  const Rsrc G = tile_rsrc(src_of(a, d.bucket) + d.grad_off + r0 * m, ext);
  const Rsrc E = tile_rsrc(a.e + d.e_off + r0 * m, a.ef ? ext : 0u);
  const Rsrc Phr = tile_rsrc(a.fac + d.ph_slot + r0 * RK, fform ? u32(rows) * RK * 4u : 0u);
  const Rsrc Qlr = tile_rsrc(a.fac + d.ql_slot, fform ? u32(m) * RK * 4u : 0u);
  const Rsrc Qhr = tile_rsrc(a.fac + d.qh_slot, u32(m) * RK * 4u);
  const bool ph4 = aligned16(a.fac + d.ph_slot), ql4 = aligned16(a.fac + d.ql_slot);
  float pa[KH];  // correction A operand: -Ph[r0 + l % 32][rk0 + KH h + s]
  load_run<KH>(Phr, u32(li * RK + rk0 + KH * h) * 4u, ph4, pa);
#pragma unroll
  for (int s = 0; s < KH; ++s) pa[s] = -pa[s];

  auto load_block = [&](int64_t c0, float* g, float* e) {  // the wave's entries
    const uint32_t coff = c0 + li < m ? u32(c0 + li) * 4u : kOut;
#pragma unroll
    for (int j = 0; j < EPW; ++j) {
      const uint32_t o = coff == kOut ? kOut : u32(drow(EPW * wave + j, h)) * row_bytes + coff;
      g[j] = bld1_nt(G, o);
      e[j] = bld1_nt(E, o);
    }
  };
  auto load_ql = [&](int64_t c0, float* qa) {  // correction B operand: Ql rows
    const int64_t qcol = c0 + li;
    load_run<KH>(Qlr, qcol < m ? u32(qcol * RK + rk0 + KH * h) * 4u : kOut, ql4, qa);
  };
  auto load_qh = [&](int64_t c0, float (*qb)[16]) {  // product B operand: Qh rows
#pragma unroll
    for (int kb = 0; kb < NR; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t col = c0 + drow(v, h);
        qb[kb][v] = bld1(Qhr, col < m ? u32(col * RK + rk0 + kb * 32 + li) * 4u : kOut);
      }
  };
  __shared__ float red[2][SW][16 * kWave];
  __shared__ float xt[2][32 * LD];
  float g[EPW], e[EPW], qa[KH], qb[NR][16];
  load_block(0, g, e);
  if (fform) load_ql(0, qa);
  load_qh(0, qb);
  v16f p[NR];
#pragma unroll
  for (int kb = 0; kb < NR; ++kb) p[kb] = zero16();
  int buf = 0;
  for (int64_t c0 = 0; c0 < m; c0 += 32, buf ^= 1) {
    // each operand's registers take the next block's values once this block has used them
    if (fform) {  // the wave's share of -Ph Ql^T: A = -Ph (row, rank), B = Ql^T (rank, column)
      v16f x = zero16();
#pragma unroll
      for (int s = 0; s < KH; ++s) x = mfma(pa[s], qa[s], x);
      load_ql(c0 + 32, qa);
#pragma unroll
      for (int v = 0; v < 16; ++v) red[buf][wave][v * kWave + lane] = x[v];
      __syncthreads();
    }
    float cg[EPW], ce[EPW];
#pragma unroll
    for (int j = 0; j < EPW; ++j) {
      cg[j] = g[j];
      ce[j] = e[j];
    }
    load_block(c0 + 32, g, e);  // next block (past m: zeros, no traffic)
    const uint32_t coff = c0 + li < m ? u32(c0 + li) * 4u : kOut;
#pragma unroll
    for (int j = 0; j < EPW; ++j) {
      const int v = EPW * wave + j, row = drow(v, h);
      float xv = cg[j] + ce[j];
      if (fform) {
        float c = red[buf][0][v * kWave + lane];
#pragma unroll
        for (int w = 1; w < SW; ++w) c += red[buf][w][v * kWave + lane];
        xv += c;
      }
      bst1_nt(E, coff == kOut ? kOut : u32(row) * row_bytes + coff, xv);
      xt[buf][row * LD + li] = xv;
    }
    __syncthreads();
#pragma unroll
    for (int v = 0; v < 16; ++v) {  // P += X Qh: A = X (row, column), B = Qh (column, rank)
      const float xa = xt[buf][li * LD + drow(v, h)];
#pragma unroll
      for (int kb = 0; kb < NR; ++kb) p[kb] = mfma(xa, qb[kb][v], p[kb]);
    }
    load_qh(c0 + 32, qb);
  }

  float* P = dst_of(a, d.bucket) + d.fac_off_p;
  float* Pl = a.fac + d.pl_slot;
#pragma unroll
  for (int kb = 0; kb < NR; ++kb) {
    const int rank = rk0 + kb * 32 + li;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int row = drow(v, h);
      if (row < rows) {
        P[(r0 + row) * RK + rank] = p[kb][v];
        Pl[(r0 + row) * RK + rank] = p[kb][v];
      }
    }
  }
}

// Q-step over a tile (row chunk t.a, 32-column block t.b), the 32-row blocks in order: partial
// corrections -Pl Qh^T (X form) -> F = M + E + their sum for the wave's entries, stored to the
// arena and shared through LDS -> Q += F^T Ph over the wave's ranks, into the chunk's partials.
template <int RK>
__global__ __launch_bounds__(kWave * split_waves(RK), 2) void k_sqstep(KArgs a) {
  constexpr int SW = split_waves(RK), EPW = 16 / SW, RS = RK / SW, KH = RS / 2, NR = RS / 32;
  static_assert(RS % 32 == 0 && EPW * SW == 16, "whole 32-rank blocks and entries per wave");
  const Tile t = a.tiles[blockIdx.x];
  const MatDesc d = a.mats[t.idx];
  const int wave = tid() >> 6, lane = tid() & 63, h = lane >> 5, li = lane & 31;
  const int rk0 = wave * RS;
  const int64_t n = d.n, m = d.m;
  const int64_t r0 = static_cast<int64_t>(t.a) * d.q_rows;
  const int rows = static_cast<int>((r0 + d.q_rows < n) ? d.q_rows : n - r0);
  const int64_t c0 = static_cast<int64_t>(t.b) * d.q_cb;
  const int64_t w = (m - c0) < 32 ? (m - c0) : 32;  // valid columns of the block
  const bool xform = deferred_p_of(a, d.bucket);
  const uint32_t row_bytes = u32(m) * 4u;
  const uint32_t ext = u32(rows - 1) * row_bytes + u32(w) * 4u;
  const Rsrc G = tile_rsrc(src_of(a, d.bucket) + d.grad_off + r0 * m + c0, ext);
  const Rsrc E = tile_rsrc(a.e + d.e_off + r0 * m + c0, a.ef ? ext : 0u);
  const Rsrc Qhr = tile_rsrc(a.fac + d.qh_slot + c0 * RK, xform ? u32(w) * RK * 4u : 0u);
  const Rsrc Plr = tile_rsrc(a.fac + d.pl_slot + r0 * RK, xform ? u32(rows) * RK * 4u : 0u);
  const Rsrc Phr = tile_rsrc(a.fac + d.ph_slot + r0 * RK, u32(rows) * RK * 4u);
  const bool qh4 = aligned16(a.fac + d.qh_slot), pl4 = aligned16(a.fac + d.pl_slot);
  float qv[KH];  // correction B operand: Qh[c0 + l % 32][rk0 + KH h + s]
  load_run<KH>(Qhr, u32(li * RK + rk0 + KH * h) * 4u, qh4, qv);
  const uint32_t coff = li < w ? u32(li) * 4u : kOut;

  auto load_block = [&](int rb, float* g, float* e) {  // the wave's entries
#pragma unroll
    for (int j = 0; j < EPW; ++j) {
      const uint32_t o = coff == kOut ? kOut : u32(rb + drow(EPW * wave + j, h)) * row_bytes + coff;
      g[j] = bld1_nt(G, o);
      e[j] = bld1_nt(E, o);
    }
  };
  auto load_ops = [&](int rb, float* pa, float (*pb)[16]) {
    if (xform) load_run<KH>(Plr, u32((rb + li) * RK + rk0 + KH * h) * 4u, pl4, pa);
#pragma unroll
    for (int kb = 0; kb < NR; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        pb[kb][v] = bld1(Phr, u32((rb + drow(v, h)) * RK + rk0 + kb * 32 + li) * 4u);
  };
  __shared__ float red[2][SW][16 * kWave];
  __shared__ float fs[2][16 * kWave];
  float g[EPW], e[EPW], pa[KH], pb[NR][16];
  load_block(0, g, e);
  load_ops(0, pa, pb);
  v16f q[NR];
#pragma unroll
  for (int kb = 0; kb < NR; ++kb) q[kb] = zero16();
  int buf = 0;
  for (int rb = 0; rb < rows; rb += 32, buf ^= 1) {
    float cg[EPW], ce[EPW], ca[KH], cb[NR][16];
#pragma unroll
    for (int j = 0; j < EPW; ++j) {
      cg[j] = g[j];
      ce[j] = e[j];
    }
#pragma unroll
    for (int s = 0; s < KH; ++s) ca[s] = pa[s];
#pragma unroll
    for (int kb = 0; kb < NR; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) cb[kb][v] = pb[kb][v];
    load_block(rb + 32, g, e);  // next block (past the chunk: zeros, no traffic)
    load_ops(rb + 32, pa, pb);
    if (xform) {  // the wave's share of -Pl Qh^T: A = -Pl (row, rank), B = Qh^T (rank, column)
      v16f x = zero16();
#pragma unroll
      for (int s = 0; s < KH; ++s) x = mfma(-ca[s], qv[s], x);
#pragma unroll
      for (int v = 0; v < 16; ++v) red[buf][wave][v * kWave + lane] = x[v];
      __syncthreads();
    }
#pragma unroll
    for (int j = 0; j < EPW; ++j) {
      const int v = EPW * wave + j;
      float f = cg[j] + ce[j];
      if (xform) {
        float c = red[buf][0][v * kWave + lane];
#pragma unroll
        for (int w2 = 1; w2 < SW; ++w2) c += red[buf][w2][v * kWave + lane];
        f += c;
      }
      bst1_nt(E, coff == kOut ? kOut : u32(rb + drow(v, h)) * row_bytes + coff, f);
      fs[buf][v * kWave + lane] = f;
    }
    __syncthreads();
#pragma unroll
    for (int v = 0; v < 16; ++v) {  // Q += F^T Ph: A = F^T, B = Ph
      const float fv = fs[buf][v * kWave + lane];
#pragma unroll
      for (int kb = 0; kb < NR; ++kb) q[kb] = mfma(fv, cb[kb][v], q[kb]);
    }
  }
  const int64_t ncb = (m + d.q_cb - 1) / d.q_cb;
  const int64_t stride = ncb * d.q_cb * RK;  // one row chunk of partials
  float* part = a.qpart + d.qpart + static_cast<int64_t>(t.a) * stride + c0 * RK;
#pragma unroll
  for (int kb = 0; kb < NR; ++kb)
#pragma unroll
    for (int v = 0; v < 16; ++v) part[drow(v, h) * RK + rk0 + kb * 32 + li] = q[kb][v];
}

// Decompress over a tile (32-row block t.a, 1024-column group t.b): per 32-column block the
// wave's share of A B^T / p, the shares added in wave order for the wave's entries and stored
// with nontemporal stores.  The next block's B rows are requested before the current MFMAs.
template <int RK>
__global__ __launch_bounds__(kWave * split_waves(RK), 2) void k_srecon(KArgs a) {
  constexpr int SW = split_waves(RK), EPW = 16 / SW, RS = RK / SW, KH = RS / 2;
  static_assert(RS % 32 == 0 && EPW * SW == 16, "whole 32-rank blocks and entries per wave");
  const Tile t = a.tiles[blockIdx.x];
  const bool odd = a.parity != 0;
  const MatDesc d = a.mats[t.idx];
  const int wave = tid() >> 6, lane = tid() & 63, h = lane >> 5, li = lane & 31;
  const int rk0 = wave * RS;
  const int64_t n = d.n, m = d.m;
  const int64_t r0 = static_cast<int64_t>(t.a) * 32;
  const int rows = static_cast<int>((r0 + 32 < n) ? 32 : n - r0);
  const float* agg = src_of(a, d.bucket);
  const float* A = odd ? agg + d.fac_off_p : a.fac + d.ph_slot;
  const float* B = odd ? a.fac + d.qh_slot : agg + d.fac_off_q;
  const Rsrc Ar = tile_rsrc(A + r0 * RK, u32(rows) * RK * 4u);
  const Rsrc Br = tile_rsrc(B, u32(m) * RK * 4u);
  const bool a4 = aligned16(A), b4 = aligned16(B);
  float av[KH];  // A operand: A[r0 + l % 32][rk0 + KH h + s] / p
  load_run<KH>(Ar, u32(li * RK + rk0 + KH * h) * 4u, a4, av);
#pragma unroll
  for (int s = 0; s < KH; ++s) av[s] *= a.inv_p;
  float* O = dst_of(a, d.bucket) + d.grad_off + r0 * m;
  const uint32_t row_bytes = u32(m) * 4u;
  constexpr int NB = kWideRCols / 32;  // column blocks per tile
  auto bcol = [&](int j) { return static_cast<int64_t>(t.b) * kWideRCols + j * 32; };
  auto boff = [&](int64_t c) { return c + li < m ? u32((c + li) * RK + rk0 + KH * h) * 4u : kOut; };
  __shared__ float red[2][SW][16 * kWave];
  float bv[2][KH];  // B operand: B[c0 + l % 32][rk0 + KH h + s], this block and the next
  load_run<KH>(Br, boff(bcol(0)), b4, bv[0]);
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int64_t c0 = bcol(j);
    if (c0 >= m) break;
    if (j + 1 < NB) load_run<KH>(Br, boff(bcol(j + 1)), b4, bv[(j + 1) & 1]);
    v16f o = zero16();
#pragma unroll
    for (int s = 0; s < KH; ++s) o = mfma(av[s], bv[j & 1][s], o);
#pragma unroll
    for (int v = 0; v < 16; ++v) red[j & 1][wave][v * kWave + lane] = o[v];
    __syncthreads();
    const int64_t w = (m - c0) < 32 ? (m - c0) : 32;
    const Rsrc Or = tile_rsrc(O + c0, u32(rows - 1) * row_bytes + u32(w) * 4u);
    const uint32_t coff = li < w ? u32(li) * 4u : kOut;
#pragma unroll
    for (int jj = 0; jj < EPW; ++jj) {
      const int v = EPW * wave + jj;
      float s = red[j & 1][0][v * kWave + lane];
#pragma unroll
      for (int w2 = 1; w2 < SW; ++w2) s += red[j & 1][w2][v * kWave + lane];
      bst1_nt(Or, coff == kOut ? kOut : u32(drow(v, h)) * row_bytes + coff, s);
    }
  }
}

// Decompress companions of K_WRECON (whole workgroups): factor tiles keep the aggregated
// factor as the next step's reused factor and build its W; vector tiles unpack sum / p.
template <int RK>
__global__ __launch_bounds__(kBlock) void k_wfact(KArgs a) {
  const Tile t = a.tiles[blockIdx.x];
  const bool odd = a.parity != 0;
  if (t.kind == T_VEC) {
    vec_tile(a, t, false);
    return;
  }
  const MatDesc d = a.mats[t.idx];
  const float* src = src_of(a, d.bucket) + (odd ? d.fac_off_p : d.fac_off_q);
  float* dst = a.fac + (odd ? d.p_slot : d.q_slot);
  fact_tile<RK>(a, t, src, dst, odd ? d.n : d.m);
}

template <int RK>
hipError_t launch_wide_rank(const Launch& l, const KArgs& args, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(l.ntiles));
  if constexpr (RK >= kSplitRank) {
    const dim3 block(kWave * split_waves(RK));
    switch (l.kernel) {
      case K_WFACT: hipLaunchKernelGGL(k_wfact<RK>, grid, dim3(kBlock), 0, s, args); break;
      case K_WPSTEP: hipLaunchKernelGGL(k_spstep<RK>, grid, block, 0, s, args); break;
      case K_WQSTEP: hipLaunchKernelGGL(k_sqstep<RK>, grid, block, 0, s, args); break;
      case K_WRECON:
        if constexpr (RK >= kSplitReconRank)
          hipLaunchKernelGGL(k_srecon<RK>, grid, block, 0, s, args);
        else
          hipLaunchKernelGGL(k_wrecon<RK>, grid, dim3(kWideBlock), 0, s, args);
        break;
      default: return hipErrorInvalidValue;
    }
  } else {
    switch (l.kernel) {
      case K_WFACT: hipLaunchKernelGGL(k_wfact<RK>, grid, dim3(kBlock), 0, s, args); break;
      case K_WPSTEP: hipLaunchKernelGGL(k_wpstep<RK>, grid, dim3(kWideBlock * kWidePWaves), 0, s, args); break;
      case K_WQSTEP: hipLaunchKernelGGL(k_wqstep<RK>, grid, dim3(kWideBlock * kWideQWaves), 0, s, args); break;
      case K_WRECON: hipLaunchKernelGGL(k_wrecon4w<RK>, grid, dim3(kBlock), 0, s, args); break;
      default: return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_wide(const Launch& l, int32_t rank, const KArgs& args, hipStream_t s) {
  if (l.ntiles <= 0) return hipSuccess;
  switch (rank) {
    case 8: return launch_wide_rank<8>(l, args, s);
    case 16: return launch_wide_rank<16>(l, args, s);
    case 32: return launch_wide_rank<32>(l, args, s);
    case 64: return launch_wide_rank<64>(l, args, s);
    case 128: return launch_wide_rank<128>(l, args, s);
    case 256: return launch_wide_rank<256>(l, args, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace acp
