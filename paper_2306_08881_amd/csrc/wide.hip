// gfx950 MFMA kernels of the ACP-SGD compressor for ranks 8, 16 and 32 (arXiv 2306.08881,
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
// Each is one rank-r correction and one rank-r product per element.
//
// MFMA layout (one wave): D (32 x 32) += A (32 x 2) B (2 x 32).  Lane l supplies
// A[l % 32][l / 32] and B[l / 32][l % 32]; register v of lane l holds D[drow(v, l / 32)][l % 32].
// The K index of a step may map to any pair of rank (or row, column) indices as long as A and
// B use the same pair; the kernels use rank (r / 2) h + s on half h at step s, and the row or
// column drow(v, h) at step v, which lets the output of one MFMA feed the next directly.
#include "device.hpp"

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

// P-step over a tile of at most 32 rows and all m columns.  Wave w takes the 32-column blocks
// w, w + 4, ...; per block, lane l holds X for row r0 + l % 32 and columns c0 + drow(v, l / 32)
// (VEC = 4: four float4 per stream, else sixteen floats).  The correction (F form) is an MFMA
// with D indexed (column, row), which leaves X in that same layout; X then is the A operand of
// P += X Qh.  The four waves' partial P are added in wave order.
template <int RK, int VEC>
__global__ __launch_bounds__(kBlock) void k_wpstep(KArgs a) {
  constexpr int KH = RK / 2;
  const Tile t = a.tiles[blockIdx.x];
  if (t.kind == T_VEC) {
    vec_tile(a, t, true);
    return;
  }
  const MatDesc d = a.mats[t.idx];
  const int wave = tid() >> 6, lane = tid() & 63, h = lane >> 5, li = lane & 31;
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
  float pv[KH];  // correction B operand: Ph[r0 + l % 32][KH h + s]
#pragma unroll
  for (int s = 0; s < KH; ++s) pv[s] = bld1(Phr, u32(li * RK + KH * h + s) * 4u);
  const uint32_t roff = u32(li) * row_bytes;  // rows past the tile fall past the extent

  v16f p = zero16();
  for (int64_t c0 = wave * 32; c0 < m; c0 += 128) {
    v16f x;
    uint32_t off[VEC == 4 ? 4 : 16];
    if constexpr (VEC == 4) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t col = c0 + 8 * q + 4 * h;
        off[q] = col < m ? roff + u32(col) * 4u : kOut;
        const float4 g = bld4_nt(G, off[q]), e = bld4_nt(E, off[q]);
        x[4 * q + 0] = g.x + e.x;
        x[4 * q + 1] = g.y + e.y;
        x[4 * q + 2] = g.z + e.z;
        x[4 * q + 3] = g.w + e.w;
      }
    } else {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t col = c0 + drow(v, h);
        off[v] = col < m ? roff + u32(col) * 4u : kOut;
        x[v] = bld1_nt(G, off[v]) + bld1_nt(E, off[v]);
      }
    }
    if (fform) {  // X -= Ph Ql^T: A = -Ql (column, rank), B = Ph^T (rank, row)
      const int64_t qcol = c0 + li;
#pragma unroll
      for (int s = 0; s < KH; ++s) {
        const float qa = -bld1(Qlr, qcol < m ? u32(qcol * RK + KH * h + s) * 4u : kOut);
        x = mfma(qa, pv[s], x);
      }
    }
    if constexpr (VEC == 4) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        bst4_nt(E, off[q], make_float4(x[4 * q], x[4 * q + 1], x[4 * q + 2], x[4 * q + 3]));
    } else {
#pragma unroll
      for (int v = 0; v < 16; ++v) bst1_nt(E, off[v], x[v]);
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) {  // P += X Qh: A = X (row, column), B = Qh (column, rank)
      const int64_t col = c0 + drow(v, h);
      const float qb = bld1(Qhr, (col < m && li < RK) ? u32(col * RK + li) * 4u : kOut);
      p = mfma(x[v], qb, p);
    }
  }

  __shared__ float red[4][32 * 32];
#pragma unroll
  for (int v = 0; v < 16; ++v) red[wave][drow(v, h) * 32 + li] = p[v];
  __syncthreads();
  float* P = dst_of(a, d.bucket) + d.fac_off_p;
  float* Pl = a.fac + d.pl_slot;
  for (int e = tid(); e < 32 * 32; e += kBlock) {
    const int row = e >> 5, k = e & 31;
    if (row < rows && k < RK) {
      const float sum = ((red[0][e] + red[1][e]) + red[2][e]) + red[3][e];
      P[(r0 + row) * RK + k] = sum;
      Pl[(r0 + row) * RK + k] = sum;
    }
  }
}

// Q-step over a tile (row chunk t.a of q_rows rows, column block t.b of 128 columns); wave w
// takes the block's columns c0 = t.b * 128 + 32 w ... c0 + 31.  Per 32-row block, lane l holds
// F for column c0 + l % 32 and rows drow(v, l / 32): coalesced 128-byte row segments.  The
// correction (X form) is an MFMA with D indexed (row, column); F then is the A operand of
// Q += F^T Ph with the rows as K.  Lane l's partial Q of column c0 + drow(v, l / 32), rank
// l % 32, goes to the chunk's partial block for K_QFIN.
template <int RK>
__global__ __launch_bounds__(kBlock) void k_wqstep(KArgs a) {
  constexpr int KH = RK / 2;
  const Tile t = a.tiles[blockIdx.x];
  if (t.kind == T_VEC) {
    vec_tile(a, t, true);
    return;
  }
  const MatDesc d = a.mats[t.idx];
  const int wave = tid() >> 6, lane = tid() & 63, h = lane >> 5, li = lane & 31;
  const int64_t n = d.n, m = d.m;
  const int64_t r0 = static_cast<int64_t>(t.a) * d.q_rows;
  const int rows = static_cast<int>((r0 + d.q_rows < n) ? d.q_rows : n - r0);
  const int64_t c0 = static_cast<int64_t>(t.b) * d.q_cb + wave * 32;
  const int64_t w = (m - c0) < 32 ? (m - c0) : 32;  // valid columns of this wave
  if (w <= 0) return;
  const bool xform = deferred_p_of(a, d.bucket);
  const uint32_t row_bytes = u32(m) * 4u;
  const uint32_t ext = u32(rows - 1) * row_bytes + u32(w) * 4u;
  const Rsrc G = tile_rsrc(src_of(a, d.bucket) + d.grad_off + r0 * m + c0, ext);
  const Rsrc E = tile_rsrc(a.e + d.e_off + r0 * m + c0, a.ef ? ext : 0u);
  const Rsrc Qhr = tile_rsrc(a.fac + d.qh_slot + c0 * RK, xform ? u32(w) * RK * 4u : 0u);
  const Rsrc Plr = tile_rsrc(a.fac + d.pl_slot + r0 * RK, xform ? u32(rows) * RK * 4u : 0u);
  const Rsrc Phr = tile_rsrc(a.fac + d.ph_slot + r0 * RK, u32(rows) * RK * 4u);
  float qv[KH];  // correction B operand: Qh[c0 + l % 32][KH h + s]
#pragma unroll
  for (int s = 0; s < KH; ++s) qv[s] = bld1(Qhr, u32(li * RK + KH * h + s) * 4u);
  const uint32_t coff = li < w ? u32(li) * 4u : kOut;

  v16f q = zero16();
  for (int rb = 0; rb < rows; rb += 32) {
    v16f x;
    uint32_t off[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      off[v] = coff == kOut ? kOut : u32(rb + drow(v, h)) * row_bytes + coff;
      x[v] = bld1_nt(G, off[v]) + bld1_nt(E, off[v]);
    }
    if (xform) {  // F -= Pl Qh^T: A = -Pl (row, rank), B = Qh^T (rank, column)
#pragma unroll
      for (int s = 0; s < KH; ++s) {
        const float pa = -bld1(Plr, u32((rb + li) * RK + KH * h + s) * 4u);
        x = mfma(pa, qv[s], x);
      }
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) bst1_nt(E, off[v], x[v]);
#pragma unroll
    for (int v = 0; v < 16; ++v) {  // Q += F^T Ph: A = F^T (column, row), B = Ph (row, rank)
      const float pb = bld1(Phr, li < RK ? u32((rb + drow(v, h)) * RK + li) * 4u : kOut);
      q = mfma(x[v], pb, q);
    }
  }
  const int64_t ncb = (m + d.q_cb - 1) / d.q_cb;
  const int64_t stride = ncb * d.q_cb * RK;  // one row chunk of partials
  float* part = a.qpart + d.qpart + static_cast<int64_t>(t.a) * stride + c0 * RK;
  if (li < RK)
#pragma unroll
    for (int v = 0; v < 16; ++v) part[drow(v, h) * RK + li] = q[v];
}

// Decompress: M_hat = A B^T / p over a tile (32-row block t.a, 512-column group t.b).  Odd
// step: A = P_agg (factor buffer), B = Qh; even step: A = Ph, B = Q_agg.  Wave w writes the
// 32-column blocks w, w + 4, ... of the group; lane l stores column c0 + l % 32 of rows
// drow(v, l / 32): two 128-byte row segments per store.  Factor tiles keep the aggregated
// factor as the next step's reused factor and build its W; vector tiles unpack sum / p.
template <int RK>
__global__ __launch_bounds__(kBlock) void k_wrecon(KArgs a) {
  constexpr int KH = RK / 2;
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
  const int wave = tid() >> 6, lane = tid() & 63, h = lane >> 5, li = lane & 31;
  const int64_t n = d.n, m = d.m;
  const int64_t r0 = static_cast<int64_t>(t.a) * 32;
  const int rows = static_cast<int>((r0 + 32 < n) ? 32 : n - r0);
  const float* agg = src_of(a, d.bucket);
  const float* A = odd ? agg + d.fac_off_p : a.fac + d.ph_slot;
  const float* B = odd ? a.fac + d.qh_slot : agg + d.fac_off_q;
  const Rsrc Ar = tile_rsrc(A + r0 * RK, u32(rows) * RK * 4u);
  const Rsrc Br = tile_rsrc(B, u32(m) * RK * 4u);
  float av[KH];  // A operand: A[r0 + l % 32][KH h + s] / p
#pragma unroll
  for (int s = 0; s < KH; ++s) av[s] = bld1(Ar, u32(li * RK + KH * h + s) * 4u) * a.inv_p;
  float* O = dst_of(a, d.bucket) + d.grad_off + r0 * m;
  const uint32_t row_bytes = u32(m) * 4u;
  for (int j = 0; j < kWideRCols / 128; ++j) {
    const int64_t c0 = static_cast<int64_t>(t.b) * kWideRCols + j * 128 + wave * 32;
    if (c0 >= m) break;
    const int64_t w = (m - c0) < 32 ? (m - c0) : 32;
    float bv[KH];  // B operand: B[c0 + l % 32][KH h + s]
#pragma unroll
    for (int s = 0; s < KH; ++s)
      bv[s] = bld1(Br, li < w ? u32((c0 + li) * RK + KH * h + s) * 4u : kOut);
    v16f o = zero16();
#pragma unroll
    for (int s = 0; s < KH; ++s) o = mfma(av[s], bv[s], o);
    const Rsrc Or = tile_rsrc(O + c0, u32(rows - 1) * row_bytes + u32(w) * 4u);
    const uint32_t coff = li < w ? u32(li) * 4u : kOut;
#pragma unroll
    for (int v = 0; v < 16; ++v)
      bst1(Or, coff == kOut ? kOut : u32(drow(v, h)) * row_bytes + coff, o[v]);
  }
}

template <int RK>
hipError_t launch_wide_rank(const Launch& l, const KArgs& args, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(l.ntiles)), block(kBlock);
  switch (l.kernel) {
    case K_WPSTEP:
      if (l.variant == 4)
        hipLaunchKernelGGL((k_wpstep<RK, 4>), grid, block, 0, s, args);
      else
        hipLaunchKernelGGL((k_wpstep<RK, 1>), grid, block, 0, s, args);
      break;
    case K_WQSTEP: hipLaunchKernelGGL(k_wqstep<RK>, grid, block, 0, s, args); break;
    case K_WRECON: hipLaunchKernelGGL(k_wrecon<RK>, grid, block, 0, s, args); break;
    default: return hipErrorInvalidValue;
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
    default: return hipErrorInvalidValue;
  }
}

}  // namespace acp
