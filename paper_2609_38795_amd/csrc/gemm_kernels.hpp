// GEMM kernels C[M,N] = A[M,K] * W[N,K]^T with fused epilogues (gfx950).
//
// bf16 path: 32x32x16 bf16 MFMA with fp32 accumulation.  Large GEMMs use the
// 256x256 ping-pong kernel over register-staged BK = 64 tiles, run
// persistently (gemm_bf16_pp64p_kernel; gemm_bf16_pp64_kernel is the same
// schedule one tile per workgroup, used for split-K); GEMMs with fewer than
// 256 such tiles use the LDS-staged gemm_bf16_kernel at 128x128 or 64x128.
// fp32 path: FMA, 64x64x16 tile.  Both hand the epilogue *pairs* of outputs:
// the value at column c and the one at column c+32, where c lies in the low
// half of a 64-column group.
// Weight rows are arranged at context creation so that every fused operation
// needs exactly such a pair: SwiGLU's gate/up values and RoPE's rotate-half
// partners (i, i + head_dim/2) land 32 columns apart in the same lane.
#pragma once

#include "device_common.hpp"

namespace alr {

// ------------------------------------------------------------------ epilogues

// Column order of the transposed V cache inside every aligned group of 16
// keys: keys 0-3, 8-11, 4-7, 12-15 (the second and third runs of four swap).
// That is the order in which the attention kernels' value MFMA consumes a
// 16-key step (lane half h supplies keys 4h..4h+3 and 8+4h..8+4h+3), so a tile
// goes from global memory to LDS unchanged.  The map is its own inverse.
__device__ __forceinline__ int vt_perm(int col) {
  return col ^ ((((col >> 2) ^ (col >> 3)) & 1) * 12);
}

// QKV projection + RoPE + key/value store.  Columns [0, H*hd) are q, then
// [H*hd, H*hd+G*hd) k, then v.  In the q and k sections, 64-column group t
// holds, in its low half, entries f = 32t .. 32t+31 of the list of
// first-half dimensions (head = f / (hd/2), i = f % (hd/2)) and, in its high
// half, their partners i + hd/2.  Outputs are written in natural order.
// The rotation of a RoPE pair (lo, hi) by (cs, sn), with its single fused
// multiply-add written out so that every epilogue form (per element, 16 rows,
// 4 columns) rounds the same way whatever contraction the compiler would pick.
__device__ __forceinline__ float rope_a(float lo, float hi, float cs, float sn) {
  return fmaf(lo, cs, -(hi * sn));
}
__device__ __forceinline__ float rope_b(float lo, float hi, float cs, float sn) {
  return fmaf(lo, sn, hi * cs);
}

// Lanes 2j and 2j+1 of an MFMA accumulator hold adjacent columns c, c+1 (c
// even) of the same rows.  Given a lane's values x_r, x_r1 of rows r and r+1,
// one DPP quad swap leaves the even lane with row r at columns c, c+1 and the
// odd lane with row r+1 at columns c, c+1, so each lane writes (or reads) two
// adjacent elements with one access instead of two.
__device__ __forceinline__ f32x2 pair_rows(int odd, float x_r, float x_r1) {
  const float x = dpp_perm<0xB1>(odd ? x_r : x_r1);
  return odd ? f32x2{x, x_r1} : f32x2{x_r, x};
}

template <typename OutT>
struct EpiQKV {
  OutT* q;            // [M, H*hd]
  OutT* k;            // row r -> k + r*kv_rs
  OutT* v;            // row r -> v + r*kv_rs (when vt_col is null)
  long kv_rs;
  const int* vt_col;  // if set: v is transposed, element (row, c) at v[c*vt_stride + vt_perm(vt_col[row])]
  long vt_stride;
  const float* cosT;  // [max_pos, hd/2]
  const float* sinT;
  const int* pos;     // (t, h, w) position of row r: pos[3 r + axis] + pos_add
  int pos_add;
  int sec0, sec01;    // frequencies < sec0 follow axis t, < sec01 axis h, the rest axis w
  int H, G, hd;
  __device__ __forceinline__ void operator()(int row, int c, float lo, float hi) const {
    const int half = hd >> 1;
    const int qd = H * hd, kd = G * hd;
    if (c < qd + kd) {
      OutT* dst;
      int cl;
      if (c < qd) {
        dst = q + (long)row * qd;
        cl = c;
      } else {
        dst = k + (long)row * kv_rs;
        cl = c - qd;
      }
      const int f = 32 * (cl >> 6) + (cl & 63);
      const int head = f / half, i = f - head * half;
      const int axis = (i < sec0) ? 0 : ((i < sec01) ? 1 : 2);
      const long p = (long)(pos[3 * row + axis] + pos_add);
      const float cs = cosT[p * half + i], sn = sinT[p * half + i];
      Elt<OutT>::st(dst + head * hd + i, rope_a(lo, hi, cs, sn));
      Elt<OutT>::st(dst + head * hd + i + half, rope_b(lo, hi, cs, sn));
    } else if (vt_col) {
      const long cl = c - qd - kd, col = vt_perm(vt_col[row]);
      Elt<OutT>::st(v + cl * vt_stride + col, lo);
      Elt<OutT>::st(v + (cl + 32) * vt_stride + col, hi);
    } else {
      OutT* dst = v + (long)row * kv_rs;
      const int cl = c - qd - kd;
      Elt<OutT>::st(dst + cl, lo);
      Elt<OutT>::st(dst + cl + 32, hi);
    }
  }
  // Columns c..c+3 and c+32..c+35 of one row (c a multiple of 4 in the low
  // half of a 64-column group), for the split-K reduce: the same arithmetic
  // per element as operator(), with 16-byte loads of the RoPE factors (the
  // four dims share a head, and an axis unless an M-RoPE section boundary
  // falls between them) and 8-byte bf16 stores.
  __device__ __forceinline__ void quad(int row, int c, const f32x4& lo, const f32x4& hi) const {
    const int half = hd >> 1;
    const int qd = H * hd, kd = G * hd;
    if (c < qd + kd) {
      OutT* dst;
      int cl;
      if (c < qd) {
        dst = q + (long)row * qd;
        cl = c;
      } else {
        dst = k + (long)row * kv_rs;
        cl = c - qd;
      }
      const int f = 32 * (cl >> 6) + (cl & 63);
      const int head = f / half, i = f - head * half;
      f32x4 cs, sn;
      const int ax0 = (i < sec0) ? 0 : ((i < sec01) ? 1 : 2);
      const int ax3 = (i + 3 < sec0) ? 0 : ((i + 3 < sec01) ? 1 : 2);
      if (ax0 == ax3) {
        const long o = (long)(pos[3 * row + ax0] + pos_add) * half + i;
        cs = *(const f32x4*)(cosT + o);
        sn = *(const f32x4*)(sinT + o);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int ie = i + e, ax = (ie < sec0) ? 0 : ((ie < sec01) ? 1 : 2);
          const long o = (long)(pos[3 * row + ax] + pos_add) * half + ie;
          cs[e] = cosT[o];
          sn[e] = sinT[o];
        }
      }
      f32x4 a, b;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a[e] = rope_a(lo[e], hi[e], cs[e], sn[e]);
        b[e] = rope_b(lo[e], hi[e], cs[e], sn[e]);
      }
      st4(dst + head * hd + i, a);
      st4(dst + head * hd + i + half, b);
    } else if (vt_col) {
#pragma unroll
      for (int e = 0; e < 4; ++e) (*this)(row, c + e, lo[e], hi[e]);
    } else {
      OutT* dst = v + (long)row * kv_rs;
      const int cl = c - qd - kd;
      st4(dst + cl, lo);
      st4(dst + cl + 32, hi);
    }
  }
  __device__ __forceinline__ static void st2(OutT* p, const f32x2& x) {
    if constexpr (std::is_same<OutT, bf16>::value)
      *(uint32_t*)p = pack2bf(x[0], x[1]);
    else
      *(f32x2*)p = x;
  }
  __device__ __forceinline__ static void st4(OutT* p, const f32x4& x) {
    if constexpr (std::is_same<OutT, bf16>::value) {
      u32x2 w;
      w[0] = pack2bf(x[0], x[1]);
      w[1] = pack2bf(x[2], x[3]);
      *(u32x2*)p = w;
    } else {
      *(f32x4*)p = x;
    }
  }
  // The 16 rows of a lane's 32-row block (row of index t: rb + 8 (t >> 2) +
  // (t & 3); rows >= M are skipped) of columns c and c+32.  Every load the
  // rows need (positions, then cos/sin, or the V^T columns) is issued before
  // any store, so the block costs two memory round trips rather than one per
  // row.  Four consecutive, 4-aligned columns of the transposed V cache go out
  // as one 8-byte store per column (bf16).
  __device__ __forceinline__ void rows16(int rb, int M, int c, const float* lo,
                                         const float* hi) const {
    const int half = hd >> 1;
    const int qd = H * hd, kd = G * hd;
    int r[16];
#pragma unroll
    for (int t = 0; t < 16; ++t) r[t] = rb + 8 * (t >> 2) + (t & 3);
    if (c < qd + kd) {
      OutT* base;
      long rs;
      int cl;
      if (c < qd) {
        base = q;
        rs = qd;
        cl = c;
      } else {
        base = k;
        rs = kv_rs;
        cl = c - qd;
      }
      const int f = 32 * (cl >> 6) + (cl & 63);
      const int head = f / half, i = f - head * half;
      const int axis = (i < sec0) ? 0 : ((i < sec01) ? 1 : 2);
      int pp[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) pp[t] = pos[3 * min(r[t], M - 1) + axis];
      float cs[16], sn[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        const long o = (long)(pp[t] + pos_add) * half + i;
        cs[t] = cosT[o];
        sn[t] = sinT[o];
      }
      // The two lanes of a column pair (i even, i+1 in the same head since half
      // is even) trade one value of each half per two rows, so the even lane
      // writes row r at i, i+1 and the odd lane row r+1: one store of two
      // elements per half instead of two single-element stores.
      const int odd = c & 1;
      float a[16], b[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        a[t] = rope_a(lo[t], hi[t], cs[t], sn[t]);
        b[t] = rope_b(lo[t], hi[t], cs[t], sn[t]);
      }
#pragma unroll
      for (int t = 0; t < 16; t += 2) {
        const f32x2 pa = pair_rows(odd, a[t], a[t + 1]), pb = pair_rows(odd, b[t], b[t + 1]);
        const int rr = r[t] + odd;
        if (rr < M) {
          OutT* dst = base + (long)rr * rs + head * hd + i - odd;
          st2(dst, pa);
          st2(dst + half, pb);
        }
      }
    } else if (vt_col) {
      const long cl = c - qd - kd;
      int col[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) col[t] = vt_col[min(r[t], M - 1)];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int t0 = 4 * g;
        if constexpr (std::is_same<OutT, bf16>::value) {
          if (r[t0 + 3] < M && col[t0 + 3] == col[t0] + 3 && (col[t0] & 3) == 0) {
            u32x2 wl, wh;
            wl[0] = pack2bf(lo[t0], lo[t0 + 1]);
            wl[1] = pack2bf(lo[t0 + 2], lo[t0 + 3]);
            wh[0] = pack2bf(hi[t0], hi[t0 + 1]);
            wh[1] = pack2bf(hi[t0 + 2], hi[t0 + 3]);
            const int pc = vt_perm(col[t0]);  // a 4-aligned run of 4 stays together
            *(u32x2*)(v + cl * vt_stride + pc) = wl;
            *(u32x2*)(v + (cl + 32) * vt_stride + pc) = wh;
            continue;
          }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (r[t0 + e] < M) {
            Elt<OutT>::st(v + cl * vt_stride + vt_perm(col[t0 + e]), lo[t0 + e]);
            Elt<OutT>::st(v + (cl + 32) * vt_stride + vt_perm(col[t0 + e]), hi[t0 + e]);
          }
      }
    } else {
      const int cl = c - qd - kd;
#pragma unroll
      for (int t = 0; t < 16; ++t)
        if (r[t] < M) {
          OutT* dst = v + (long)r[t] * kv_rs;
          Elt<OutT>::st(dst + cl, lo[t]);
          Elt<OutT>::st(dst + cl + 32, hi[t]);
        }
    }
  }
};

// Epilogues that read memory, or that write two columns per access, define
// rows16(): a lane's 16 rows of a 32-row block at once, all loads before all
// stores (the compiler cannot prove that a later row's load does not alias an
// earlier row's store, so element-wise calls would wait for one load round
// trip per row).
template <class Epi, class = void>
struct has_rows16 : std::false_type {};
template <class Epi>
struct has_rows16<Epi, decltype((void)&Epi::rows16)> : std::true_type {};

// Residual add into the fp32 stream, optionally capturing the new value as a
// feature row: feat + (perm ? perm[row] : row) * feat_rs.
struct EpiResid {
  float* h;
  int ld;
  float* feat;
  long feat_rs;
  const int* perm;
  __device__ __forceinline__ void operator()(int row, int c, float lo, float hi) const {
    float* p = h + (long)row * ld + c;
    const float a = p[0] + lo, b = p[32] + hi;
    p[0] = a;
    p[32] = b;
    if (feat) {
      const long r = perm ? perm[row] : row;
      float* f = feat + r * feat_rs + c;
      f[0] = a;
      f[32] = b;
    }
  }
  // Without feature rows all 16 rows' loads are issued before the first store,
  // so a wave waits one memory round trip per 32-row block instead of one per
  // 8 rows (the whole workgroup reaches its epilogue together, and those waits
  // leave the CU's matrix cores idle).  With feature rows (and their
  // permutation indices) two halves of 8 rows bound the registers the
  // epilogue needs inside a persistent kernel.
  __device__ __forceinline__ void rows16(int rb, int M, int c, const float* lo,
                                         const float* hi) const {
    if (!feat) {
      float a[16], b[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        const int rc = min(rb + 8 * (t >> 2) + (t & 3), M - 1);
        const float* p = h + (long)rc * ld + c;
        a[t] = p[0];
        b[t] = p[32];
      }
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        const int r = rb + 8 * (t >> 2) + (t & 3);
        if (r < M) {
          float* p = h + (long)r * ld + c;
          p[0] = a[t] + lo[t];
          p[32] = b[t] + hi[t];
        }
      }
      return;
    }
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      int fr[8];
      float a[8], b[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int t = 8 * half + u;
        const int r = rb + 8 * (t >> 2) + (t & 3), rc = min(r, M - 1);
        const float* p = h + (long)rc * ld + c;
        a[u] = p[0];
        b[u] = p[32];
        fr[u] = perm ? perm[rc] : r;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int t = 8 * half + u;
        const int r = rb + 8 * (t >> 2) + (t & 3);
        if (r < M) {
          a[u] += lo[t];
          b[u] += hi[t];
          float* p = h + (long)r * ld + c;
          p[0] = a[u];
          p[32] = b[u];
          float* f = feat + (long)fr[u] * feat_rs + c;
          f[0] = a[u];
          f[32] = b[u];
        }
      }
    }
  }
};

// SwiGLU: 64-column group t holds gate rows 32t..32t+31 then up rows
// 32t..32t+31; out[row, 32t + w] = SiLU(gate) * up.
template <typename OutT>
struct EpiSwiGLU {
  OutT* out;
  int ld;
  // SiLU(g) = g / (1 + e^-g) with the hardware exp2 and reciprocal (about
  // 2 ulp of fp32; e^-g overflowing to inf gives the limit 0), times u
  __device__ static __forceinline__ float act(float g, float u) {
    const float s = g * __builtin_amdgcn_rcpf(1.0f + fast_exp2(-1.44269504088896341f * g));
    return s * u;
  }
  __device__ __forceinline__ void operator()(int row, int c, float g, float u) const {
    const int col = (c >> 6) * 32 + (c & 63);
    Elt<OutT>::st(out + (long)row * ld + col, act(g, u));
  }
  // Rows rb + 8 q + e of one column, written two columns per store after the
  // lane-pair exchange (pair_rows); the pair's first output column is even
  // because d_ffn is a multiple of 64.
  __device__ __forceinline__ void rows16(int rb, int M, int c, const float* lo,
                                         const float* hi) const {
    const int odd = c & 1;
    const int col = (c >> 6) * 32 + (c & 63) - odd;
    float y[16];
#pragma unroll
    for (int t = 0; t < 16; ++t) y[t] = act(lo[t], hi[t]);
#pragma unroll
    for (int t = 0; t < 16; t += 2) {
      const f32x2 x = pair_rows(odd, y[t], y[t + 1]);
      const int r = rb + 8 * (t >> 2) + (t & 3) + odd;
      if (r < M) {
        if constexpr (std::is_same<OutT, bf16>::value)
          *(uint32_t*)(out + (long)r * ld + col) = pack2bf(x[0], x[1]);
        else
          *(f32x2*)(out + (long)r * ld + col) = x;
      }
    }
  }
};

// Per-row statistics of the output-head logits over one 64-column group: the
// group's max m and s = sum of exp(z - m) over its 64 entries.  The
// finalisation merges a row's groups into its log-sum-exp without another pass
// over the logits (and finds the lowest column holding the max in its one pass).
struct LogitPart {
  float m, s;
};

// LogitPart of one row over the 64-column group held by a 32-lane half-wave:
// lane lr of the half holds column 64 g + lr (lo) and that + 32 (hi).  Every
// lane of the half must call this with the same row; the result is the same
// in all of them.
__device__ __forceinline__ LogitPart half_wave_part(float lo, float hi) {
  float mx = group_max<16>(fmaxf(lo, hi));
  mx = max_xor16(mx);
  const float l2e = 1.44269504088896341f;
  float e = fast_exp2((lo - mx) * l2e) + fast_exp2((hi - mx) * l2e);
  e = sum_xor16(group_sum<16>(e));
  return {mx, e};
}

// fp32 logits into caller rows: out + (perm ? perm[row] : row) * rs; with part,
// also the row's LogitPart of each 64-column group into part[row * part_ld + c / 64].
// Every call site hands a 64-column group of one row to one 32-lane half-wave
// (gemm_store_tile, gemm_f32_kernel), which the partials rely on; split-K is
// not used for this epilogue when part is set.
struct EpiLogits {
  float* out;
  long rs;
  const int* perm;
  LogitPart* part;
  int part_ld;
  __device__ __forceinline__ void operator()(int row, int c, float lo, float hi) const {
    const long r = perm ? perm[row] : row;
    float* p = out + r * rs + c;
    p[0] = lo;
    p[32] = hi;
    if (part) {
      const LogitPart q = half_wave_part(lo, hi);
      if ((threadIdx.x & 31) == 0) part[(long)row * part_ld + (c >> 6)] = q;
    }
  }
  __device__ __forceinline__ void rows16(int rb, int M, int c, const float* lo,
                                         const float* hi) const {
    int rr[16];
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      const int r = rb + 8 * (t >> 2) + (t & 3);
      rr[t] = perm ? perm[min(r, M - 1)] : r;
    }
#pragma unroll
    for (int t = 0; t < 16; ++t)
      if (rb + 8 * (t >> 2) + (t & 3) < M) {
        float* p = out + (long)rr[t] * rs + c;
        p[0] = lo[t];
        p[32] = hi[t];
      }
    if (part) {
      // all 16 rows reduced over the half-wave; lane lr < 16 then stores row t = lr
      const int lr = threadIdx.x & 31;
      LogitPart mine = {0.f, 0.f};
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        const LogitPart q = half_wave_part(lo[t], hi[t]);
        if (lr == t) mine = q;
      }
      const int r = rb + 8 * (lr >> 2) + (lr & 3);
      if (lr < 16 && r < M) part[(long)r * part_ld + (c >> 6)] = mine;
    }
  }
};

// Epilogue of a wave's MI x NI block of 32x32 accumulators whose top-left
// output is (row0, col0): lane (lr, lh) of block (mi, nj) holds rows row0 +
// 32 mi + 8 q + 4 lh + e (q, e = 0..3; register 4 q + e) of columns col0 +
// 64 nj + lr and that + 32 (accumulators 2 nj and 2 nj + 1).  Epilogues with
// a rows16() form get those 16 rows in one call.
template <int MI, int NI, class Epi>
__device__ __forceinline__ void gemm_store_tile(const Epi& epi, const f32x16 (&acc)[MI][NI],
                                                int row0, int col0, int M, int N) {
  const int lane = threadIdx.x & 63, lr = lane & 31, lh = lane >> 5;
#pragma unroll
  for (int nj = 0; nj < NI / 2; ++nj) {
    const int col = col0 + nj * 64 + lr;
    if (col < N) {
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) {
        if constexpr (has_rows16<Epi>::value) {
          const int rb = row0 + mi * 32 + 4 * lh;
          if (rb < M) {
            float lo[16], hi[16];
#pragma unroll
            for (int t = 0; t < 16; ++t) {
              lo[t] = acc[mi][2 * nj][t];
              hi[t] = acc[mi][2 * nj + 1][t];
            }
            epi.rows16(rb, M, col, lo, hi);
          }
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int row = row0 + mi * 32 + 8 * q + 4 * lh;
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (row + e < M) epi(row + e, col, acc[mi][2 * nj][4 * q + e], acc[mi][2 * nj + 1][4 * q + e]);
          }
        }
      }
    }
  }
}

// Split-K: slice s of the K range writes raw fp32 sums of columns c and c+32
// to out + s * sstride + row * ld; splitk_reduce_kernel adds the slices in
// slice order (the result does not depend on which slice finished first) and
// applies the real epilogue.
struct EpiPartial {
  float* out;
  long sstride;
  int ld;
  __device__ __forceinline__ void set_split(int sl) { out += sl * sstride; }
  __device__ __forceinline__ void operator()(int row, int c, float lo, float hi) const {
    out[(long)row * ld + c] = lo;
    out[(long)row * ld + c + 32] = hi;
  }
};

template <class Epi, class = void>
struct has_set_split : std::false_type {};
template <class Epi>
struct has_set_split<Epi, decltype((void)&Epi::set_split)> : std::true_type {};

// One thread per (row, column c in the low half of a 64-column group).  With
// S > 0 the slice count is S and every partial is loaded before the first add:
// one memory round trip, where a load followed by its add in a loop over a
// runtime count has the compiler wait in every iteration.  S = 0 reads
// `slices` partials in such a loop.  Either way the slices are added in slice
// order, so the result does not depend on S.
template <class Epi, int S = 0>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part,
                                                            long sstride, int slices, int M,
                                                            int N, Epi epi) {
  const long t = (long)blockIdx.x * 256 + threadIdx.x;
  const int groups = N / 64;
  if (t >= (long)M * groups * 32) return;
  const int c32 = (int)(t & 31);
  const long rg = t >> 5;
  const int g = (int)(rg % groups), row = (int)(rg / groups);
  const int col = g * 64 + c32;
  const float* p = part + (long)row * N + col;
  float lo = 0.f, hi = 0.f;
  if constexpr (S > 0) {
    float a[S], b[S];
#pragma unroll
    for (int sl = 0; sl < S; ++sl) {
      a[sl] = p[sl * sstride];
      b[sl] = p[sl * sstride + 32];
    }
#pragma unroll
    for (int sl = 0; sl < S; ++sl) {
      lo += a[sl];
      hi += b[sl];
    }
  } else {
    for (int sl = 0; sl < slices; ++sl) {
      lo += p[sl * sstride];
      hi += p[sl * sstride + 32];
    }
  }
  epi(row, col, lo, hi);
}

template <class Epi, class = void>
struct has_quad : std::false_type {};
template <class Epi>
struct has_quad<Epi, decltype((void)&Epi::quad)> : std::true_type {};

// splitk_reduce_kernel for epilogues with quad(): one thread per (row, 4-column
// run in the low half of a 64-column group) with 16-byte partial loads; each
// element is summed in slice order as there.
template <class Epi, int S>
__global__ __launch_bounds__(256) void splitk_reduce4_kernel(const float* __restrict__ part,
                                                             long sstride, int M, int N, Epi epi) {
  const long t = (long)blockIdx.x * 256 + threadIdx.x;
  const int groups = N / 64;
  if (t >= (long)M * groups * 8) return;
  const int c4 = (int)(t & 7);
  const long rg = t >> 3;
  const int g = (int)(rg % groups), row = (int)(rg / groups);
  const int col = g * 64 + 4 * c4;
  const float* p = part + (long)row * N + col;
  f32x4 a[S], b[S];
#pragma unroll
  for (int sl = 0; sl < S; ++sl) {
    a[sl] = *(const f32x4*)(p + sl * sstride);
    b[sl] = *(const f32x4*)(p + sl * sstride + 32);
  }
  f32x4 lo, hi;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    lo[e] = 0.f;
    hi[e] = 0.f;
  }
#pragma unroll
  for (int sl = 0; sl < S; ++sl)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lo[e] += a[sl][e];
      hi[e] += b[sl][e];
    }
  epi.quad(row, col, lo, hi);
}

// ------------------------------------------------------------------ bf16 MFMA GEMM
//
// Workgroup tile BM x BN, WGM x WGN waves, wave tile (BM/WGM) x (BN/WGN) with a
// width that is a multiple of 64 so the epilogue pairs c and c+32 sit in one
// lane.
// K is consumed in steps of BK through two LDS stages.  Global loads run two
// steps ahead into two register sets; the steady-state loop handles two steps
// per iteration with no data-dependent branches (prefetch offsets are clamped
// to the last step, so the final iterations re-read it harmlessly), which
// keeps the compiler's wait counting exact.  Within a step the LDS fragments
// of k-slice ks+1 are read while the MFMAs of slice ks run.  LDS rows of BK
// bf16 are XOR-swizzled in 16-byte chunks so ds_read_b128 / ds_write_b128 are
// free of bank conflicts.

// Tile order: workgroups are dispatched round-robin over the 8 XCDs, so the
// block id is first remapped to make each XCD walk a contiguous range of the
// tile order; the order itself groups 8 M-tiles per N sweep so neighbouring
// tiles share A rows and W rows in L2.
__device__ __forceinline__ void gemm_tile_coords(int bid, int tiles_m, int tiles_n, int& tm,
                                                 int& tn) {
  const int nb = tiles_m * tiles_n;
  if ((nb & 7) == 0) bid = (bid & 7) * (nb >> 3) + (bid >> 3);
  const int group = 8;
  const int per_group = group * tiles_n;
  const int g = bid / per_group;
  const int first_m = g * group;
  const int gm = min(tiles_m - first_m, group);
  const int in = bid - g * per_group;
  tm = first_m + in % gm;
  tn = in / gm;
}
__device__ __forceinline__ void gemm_tile_coords(int tiles_m, int tiles_n, int& tm, int& tn) {
  gemm_tile_coords(blockIdx.x, tiles_m, tiles_n, tm, tn);
}

// Element offset of 16-byte chunk c of LDS row r for rows of BK bf16.
//  BK = 32 (4 chunks, 64 B): h = ((r>>2)&1)<<1 | ((r>>1)^(r>>3))&1
//  BK = 64 (8 chunks, 128 B): h = (r & 7) ^ ((r >> 3) & 1)
// Either way the 16 rows a 16-lane group reads with one ds_read_b128 cover all
// 16 granules of a 256-byte LDS line, and 8 aligned rows cover the 8
// granules of a 128-byte line.
template <int BK>
__device__ __forceinline__ int swz(int r, int c) {
  if constexpr (BK == 32) {
    const int h = (((r >> 2) & 1) << 1) | (((r >> 1) ^ (r >> 3)) & 1);
    return r * 32 + ((c ^ h) << 3);
  } else {
    const int h = (r & 7) ^ ((r >> 3) & 1);
    return r * 64 + ((c ^ h) << 3);
  }
}

template <int CH>
struct GemmRegs {
  u32x4 v[CH];
};

template <int CH>
__device__ __forceinline__ void gemm_gload(GemmRegs<CH>& r, const bf16* const* src, int ko) {
#pragma unroll
  for (int i = 0; i < CH; ++i) r.v[i] = *(const u32x4*)(src[i] + ko);
}

template <int CH>
__device__ __forceinline__ void gemm_lstore(const GemmRegs<CH>& r, bf16* stage, const int* off) {
#pragma unroll
  for (int i = 0; i < CH; ++i) *(u32x4*)(stage + off[i]) = r.v[i];
}

template <int MI, int NI>
struct GemmFrag {
  bf16x8 a[MI], b[NI];
};

template <int BK, int MI, int NI, int WTM, int WTN>
__device__ __forceinline__ void gemm_frag_load(GemmFrag<MI, NI>& f, const bf16* As,
                                               const bf16* Ws, int wm, int wn, int ks) {
  const int lane = threadIdx.x & 63, lr = lane & 31, lh = lane >> 5;
  const int c = ks * 2 + lh;
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
    f.a[mi] = as_bf16x8(*(const u32x4*)(As + swz<BK>(wm * WTM + mi * 32 + lr, c)));
#pragma unroll
  for (int ni = 0; ni < NI; ++ni)
    f.b[ni] = as_bf16x8(*(const u32x4*)(Ws + swz<BK>(wn * WTN + ni * 32 + lr, c)));
}

template <int MI, int NI>
__device__ __forceinline__ void gemm_frag_mma(const GemmFrag<MI, NI>& f,
                                              f32x16 (&acc)[MI][NI]) {
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) acc[mi][ni] = mfma32x32x16(f.a[mi], f.b[ni], acc[mi][ni]);
}

// MFMAs of one LDS stage, k-slice by k-slice, reading the fragments of slice
// ks+1 while slice ks runs, and writing the next step's operand registers
// (ra, rw) into the other LDS stage a few chunks per slice so the LDS writes
// overlap the MFMAs instead of bunching up before the barrier.
template <int BK, int MI, int NI, int WTM, int WTN, int A_CH, int W_CH>
__device__ __forceinline__ void gemm_stage_mma(const bf16* As, const bf16* Ws, int wm, int wn,
                                               f32x16 (&acc)[MI][NI], const GemmRegs<A_CH>& ra,
                                               const GemmRegs<W_CH>& rw, bf16* As_nx, bf16* Ws_nx,
                                               const int* a_off, const int* w_off) {
  constexpr int KS = BK / 16;
  GemmFrag<MI, NI> f[2];
  gemm_frag_load<BK, MI, NI, WTM, WTN>(f[0], As, Ws, wm, wn, 0);
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    if (ks + 1 < KS) gemm_frag_load<BK, MI, NI, WTM, WTN>(f[(ks + 1) & 1], As, Ws, wm, wn, ks + 1);
    gemm_frag_mma<MI, NI>(f[ks & 1], acc);
#pragma unroll
    for (int i = 0; i < A_CH; ++i)
      if (i % KS == ks) *(u32x4*)(As_nx + a_off[i]) = ra.v[i];
#pragma unroll
    for (int i = 0; i < W_CH; ++i)
      if (i % KS == ks) *(u32x4*)(Ws_nx + w_off[i]) = rw.v[i];
    __builtin_amdgcn_sched_barrier(0);  // keep each slice's writes with its MFMAs
  }
}

// TAG only separates the instantiations of different call sites, so that
// profilers report each GEMM of the model on its own line.  K must be a
// multiple of 2*BK.  With splits > 1 (an epilogue with set_split) workgroup b
// computes K slice b % splits of tile b / splits, K being the slice length.
template <int TAG, int BM, int BN, int WGM, int WGN, int BK, int OCC, class Epi>
__global__ __launch_bounds__(64 * WGM * WGN, OCC) void gemm_bf16_kernel(
    const bf16* __restrict__ A, int lda, const bf16* __restrict__ W, int ldw, int M, int N, int K,
    int tiles_m, int tiles_n, Epi epi, int splits = 1) {
  constexpr int NT = 64 * WGM * WGN;  // threads
  constexpr int WTM = BM / WGM;  // wave tile rows
  constexpr int WTN = BN / WGN;  // wave tile columns (multiple of 64: epilogue pairs c, c+32)
  static_assert(WTN % 64 == 0, "wave tile width must be a multiple of 64");
  constexpr int MI = WTM / 32;   // 32x32 blocks per wave along M
  constexpr int NI = WTN / 32;   // and along N
  constexpr int CPR = BK / 8;    // 16-byte chunks per row
  constexpr int A_CH = BM * CPR / NT, W_CH = BN * CPR / NT;  // chunks per thread
  static_assert(A_CH >= 1 && W_CH >= 1 && A_CH * NT == BM * CPR && W_CH * NT == BN * CPR,
                "tile does not split evenly over the threads");
  __shared__ __attribute__((aligned(16))) bf16 As[2][BM * BK];
  __shared__ __attribute__((aligned(16))) bf16 Ws[2][BN * BK];

  int bid = blockIdx.x;
  if constexpr (has_set_split<Epi>::value) {
    if (splits > 1) {
      const int sl = bid % splits;
      bid /= splits;
      A += (long)sl * K;
      W += (long)sl * K;
      epi.set_split(sl);
    }
  }
  int tm, tn;
  gemm_tile_coords(bid, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;

  const bf16* a_src[A_CH];
  const bf16* w_src[W_CH];
  int a_off[A_CH], w_off[W_CH];
#pragma unroll
  for (int i = 0; i < A_CH; ++i) {
    const int ch = tid + NT * i, r = ch / CPR, c = ch % CPR;
    a_src[i] = A + (long)min(m0 + r, M - 1) * lda + c * 8;
    a_off[i] = swz<BK>(r, c);
  }
#pragma unroll
  for (int i = 0; i < W_CH; ++i) {
    const int ch = tid + NT * i, r = ch / CPR, c = ch % CPR;
    w_src[i] = W + (long)min(n0 + r, N - 1) * ldw + c * 8;
    w_off[i] = swz<BK>(r, c);
  }
  const int nk = K / BK;  // even, >= 2
  const int klast = (nk - 1) * BK;

  GemmRegs<A_CH> ra0, ra1;
  GemmRegs<W_CH> rw0, rw1;
  gemm_gload(ra0, a_src, 0);
  gemm_gload(rw0, w_src, 0);
  gemm_gload(ra1, a_src, BK);
  gemm_gload(rw1, w_src, BK);
  gemm_lstore(ra0, As[0], a_off);
  gemm_lstore(rw0, Ws[0], w_off);
  __syncthreads();

  f32x16 acc[MI][NI];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < NI; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.f;

  for (int kt = 0; kt < nk; kt += 2) {
    // step kt from stage 0; set 0 refills with step kt+2; set 1 (step kt+1) -> stage 1
    const int k2 = min((kt + 2) * BK, klast), k3 = min((kt + 3) * BK, klast);
    gemm_gload(ra0, a_src, k2);
    gemm_gload(rw0, w_src, k2);
    __builtin_amdgcn_sched_barrier(0);  // keep the prefetch at the top of the step
    gemm_stage_mma<BK, MI, NI, WTM, WTN, A_CH, W_CH>(As[0], Ws[0], wm, wn, acc, ra1, rw1, As[1],
                                                     Ws[1], a_off, w_off);
    __syncthreads();
    // step kt+1 from stage 1; set 1 refills with step kt+3; set 0 (step kt+2) -> stage 0
    gemm_gload(ra1, a_src, k3);
    gemm_gload(rw1, w_src, k3);
    __builtin_amdgcn_sched_barrier(0);
    gemm_stage_mma<BK, MI, NI, WTM, WTN, A_CH, W_CH>(As[1], Ws[1], wm, wn, acc, ra0, rw0, As[0],
                                                     Ws[0], a_off, w_off);
    __syncthreads();
  }

  gemm_store_tile<MI, NI>(epi, acc, m0 + wm * WTM, n0 + wn * WTN, M, N);
}

// ------------------------------------------------------------------ bf16 MFMA GEMM, ping-pong, BK = 64
//
// 256x256 tile, 8 waves, two LDS stages of BK = 64 (rows of 128 bytes, so every
// global request is a whole cache line).  Groups as in gemm_bf16_pp_kernel
// (waves w and w+4 share a SIMD; group g owns rows [128 g, 128 g + 128)).  A
// step is consumed in two half-steps u = 2s + h (k-slices 2h, 2h+1), each a
// memory phase then a compute phase per group, group 1 one phase behind.
//
// Memory phase of half-step (s, h): read this half-step's fragments from
// stage s % 2; write the registers holding half h of step s+1 (h = 0: A rows,
// h = 1: W rows) into stage (s+1) % 2; load half h of step s+2 into the same
// registers.  Loads therefore have one step of latency cover, and a stage is
// rewritten only after both groups finished reading it (the barrier after the
// last memory phase of step s-1).  Each memory phase ends with its LDS work
// complete, so the barrier publishes the writes.
// With splits > 1 the grid holds `splits` workgroups per tile: workgroup b
// computes K slice b % splits (K is then the slice length; A and W advance by
// slice * K columns) of tile b / splits, for an epilogue with set_split.
template <int TAG, class Epi>
__global__ __launch_bounds__(512, 1) void gemm_bf16_pp64_kernel(
    const bf16* __restrict__ A, int lda, const bf16* __restrict__ W, int ldw, int M, int N, int K,
    int tiles_m, int tiles_n, Epi epi, int splits = 1) {
  constexpr int BM = 256, BN = 256, BK = 64;
  constexpr int WTM = 128, WTN = 64, MI = 4, NI = 2;
  constexpr int STAGE = (BM + BN) * BK;  // bf16 elements
  __shared__ __attribute__((aligned(1024))) bf16 smem[2 * STAGE];

  int bid = blockIdx.x;
  if constexpr (has_set_split<Epi>::value) {
    if (splits > 1) {
      const int sl = bid % splits;
      bid /= splits;
      A += (long)sl * K;
      W += (long)sl * K;
      epi.set_split(sl);
    }
  }
  int tm, tn;
  gemm_tile_coords(bid, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;
  const int wm = grp, wn = wave & 3;

  // half 0 = the A tile (256 rows x 8 chunks), half 1 = the W tile; thread t
  // moves chunks t + 512 i, i = 0..3, of each half.
  uint32_t goff[2][4];
  int loff[2][4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ch = tid + 512 * i, r = ch >> 3, c = ch & 7;
    goff[0][i] = (uint32_t)(((long)min(m0 + r, M - 1) * lda + c * 8) * 2);
    goff[1][i] = (uint32_t)(((long)min(n0 + r, N - 1) * ldw + c * 8) * 2);
    loff[0][i] = swz<BK>(r, c);
    loff[1][i] = BM * BK + swz<BK>(r, c);
  }
  const int nk = K / BK;
  const char* gbase[2] = {(const char*)A, (const char*)W};
  auto gload = [&](GemmRegs<4>& rg, int h, int step) {
    const char* b = gbase[h] + (long)min(step, nk - 1) * BK * 2;
#pragma unroll
    for (int i = 0; i < 4; ++i) rg.v[i] = *(const u32x4*)(b + goff[h][i]);
  };
  auto lstore = [&](const GemmRegs<4>& rg, int h, bf16* stage) {
#pragma unroll
    for (int i = 0; i < 4; ++i) *(u32x4*)(stage + loff[h][i]) = rg.v[i];
  };

  GemmRegs<4> rg[2];
  gload(rg[0], 0, 0);
  gload(rg[1], 1, 0);
  lstore(rg[0], 0, smem);
  lstore(rg[1], 1, smem);
  gload(rg[0], 0, 1);
  gload(rg[1], 1, 1);
  __syncthreads();
  if (grp == 1) __builtin_amdgcn_s_barrier();  // group 1 runs one phase behind

  f32x16 acc[MI][NI];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < NI; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.f;

  GemmFrag<MI, NI> f0, f1;
  for (int kt = 0; kt < nk; ++kt) {
    const bf16* cur = smem + (kt & 1) * STAGE;
    bf16* nxt = smem + ((kt + 1) & 1) * STAGE;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      // memory phase
      __builtin_amdgcn_sched_barrier(0);
      gemm_frag_load<BK, MI, NI, WTM, WTN>(f0, cur, cur + BM * BK, wm, wn, 2 * h);
      gemm_frag_load<BK, MI, NI, WTM, WTN>(f1, cur, cur + BM * BK, wm, wn, 2 * h + 1);
      lstore(rg[h], h, nxt);
      gload(rg[h], h, kt + 2);
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): fragments read, stage writes done
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      // compute phase
      __builtin_amdgcn_s_setprio(1);
      gemm_frag_mma<MI, NI>(f0, acc);
      gemm_frag_mma<MI, NI>(f1, acc);
      __builtin_amdgcn_s_setprio(0);
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_barrier();
    }
  }
  if (grp == 0) __builtin_amdgcn_s_barrier();

  gemm_store_tile<MI, NI>(epi, acc, m0 + wm * WTM, n0 + wn * WTN, M, N);
}

// ------------------------------------------------------------------ bf16 MFMA GEMM, ping-pong, persistent
//
// gemm_bf16_pp64_kernel's schedule run by one workgroup per CU over tiles
// blockIdx.x, blockIdx.x + gridDim.x, ...  The k-steps of consecutive tiles
// form one stream: in the last two k-steps of a tile the global loads already
// fetch the next tile's first two steps, and the LDS stage parity runs on
// across tiles.  A group's epilogue sits between its last compute phase of a
// tile and its first memory phase of the next, i.e. while the other group
// computes, so the pipeline is neither drained nor refilled between tiles.
template <int TAG, class Epi>
__global__ __launch_bounds__(512, 1) void gemm_bf16_pp64p_kernel(
    const bf16* __restrict__ A, int lda, const bf16* __restrict__ W, int ldw, int M, int N, int K,
    int tiles_m, int tiles_n, Epi epi) {
  constexpr int BM = 256, BN = 256, BK = 64;
  constexpr int WTM = 128, WTN = 64, MI = 4, NI = 2;
  constexpr int STAGE = (BM + BN) * BK;  // bf16 elements
  __shared__ __attribute__((aligned(1024))) bf16 smem[2 * STAGE];

  const int ntiles = tiles_m * tiles_n;
  int tile = blockIdx.x;
  if (tile >= ntiles) return;  // uniform over the workgroup
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;
  const int wm = grp, wn = wave & 3;
  const int nk = K / BK;

  // thread t moves chunks t + 512 i (row ch >> 3, 16-byte chunk ch & 7) of
  // the A tile (half 0) and of the W tile (half 1)
  int loff[2][4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ch = tid + 512 * i, r = ch >> 3, c = ch & 7;
    loff[0][i] = swz<BK>(r, c);
    loff[1][i] = BM * BK + swz<BK>(r, c);
  }
  auto offsets = [&](int t, uint32_t (&go)[2][4]) {
    int tm, tn;
    gemm_tile_coords(t, tiles_m, tiles_n, tm, tn);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ch = tid + 512 * i, r = ch >> 3, c = ch & 7;
      go[0][i] = (uint32_t)(((long)min(tm * BM + r, M - 1) * lda + c * 8) * 2);
      go[1][i] = (uint32_t)(((long)min(tn * BN + r, N - 1) * ldw + c * 8) * 2);
    }
  };
  uint32_t gcur[2][4], gnxt[2][4];
  int next = tile + gridDim.x;
  offsets(tile, gcur);
  offsets(next < ntiles ? next : tile, gnxt);
  const char* gbase[2] = {(const char*)A, (const char*)W};
  // step s of the stream relative to the current tile: s < nk is the current
  // tile, s >= nk the next one (or the current tile's last step when there is
  // none; those loads are never used)
  auto gload = [&](GemmRegs<4>& rg, int h, int s) {
    const bool nx = s >= nk;
    const int st = nx ? (next < ntiles ? s - nk : nk - 1) : s;
    const char* b = gbase[h] + (long)st * BK * 2;
#pragma unroll
    for (int i = 0; i < 4; ++i) rg.v[i] = *(const u32x4*)(b + (nx ? gnxt[h][i] : gcur[h][i]));
  };
  auto lstore = [&](const GemmRegs<4>& rg, int h, bf16* stage) {
#pragma unroll
    for (int i = 0; i < 4; ++i) *(u32x4*)(stage + loff[h][i]) = rg.v[i];
  };

  GemmRegs<4> rg[2];
  gload(rg[0], 0, 0);
  gload(rg[1], 1, 0);
  lstore(rg[0], 0, smem);
  lstore(rg[1], 1, smem);
  gload(rg[0], 0, 1);
  gload(rg[1], 1, 1);
  __syncthreads();
  if (grp == 1) __builtin_amdgcn_s_barrier();  // group 1 runs one phase behind

  f32x16 acc[MI][NI];
  GemmFrag<MI, NI> f0, f1;
  int gs = 0;  // k-steps done by this workgroup over all its tiles
  while (true) {
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < NI; ++ni)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.f;
    for (int kt = 0; kt < nk; ++kt, ++gs) {
      const bf16* cur = smem + (gs & 1) * STAGE;
      bf16* nxt = smem + ((gs + 1) & 1) * STAGE;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        // memory phase
        __builtin_amdgcn_sched_barrier(0);
        gemm_frag_load<BK, MI, NI, WTM, WTN>(f0, cur, cur + BM * BK, wm, wn, 2 * h);
        gemm_frag_load<BK, MI, NI, WTM, WTN>(f1, cur, cur + BM * BK, wm, wn, 2 * h + 1);
        lstore(rg[h], h, nxt);
        gload(rg[h], h, kt + 2);
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): fragments read, stage writes done
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        // compute phase
        __builtin_amdgcn_s_setprio(1);
        gemm_frag_mma<MI, NI>(f0, acc);
        gemm_frag_mma<MI, NI>(f1, acc);
        __builtin_amdgcn_s_setprio(0);
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_barrier();
      }
    }
    int tm, tn;
    gemm_tile_coords(tile, tiles_m, tiles_n, tm, tn);
    gemm_store_tile<MI, NI>(epi, acc, tm * BM + wm * WTM, tn * BN + wn * WTN, M, N);
    if (next >= ntiles) break;
    tile = next;
    next = tile + gridDim.x;
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int i = 0; i < 4; ++i) gcur[hh][i] = gnxt[hh][i];
    if (next < ntiles) offsets(next, gnxt);
  }
  if (grp == 0) __builtin_amdgcn_s_barrier();
}

// ------------------------------------------------------------------ fp32 FMA GEMM

constexpr int GF_M = 64, GF_N = 64, GF_K = 16;

template <int TAG, class Epi>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A, int lda,
                                                       const float* __restrict__ W, int ldw,
                                                       int M, int N, int K, int tiles_m,
                                                       int tiles_n, Epi epi) {
  __shared__ float As[GF_K][GF_M + 4];
  __shared__ float Ws[GF_K][GF_N + 4];
  int tm, tn;
  gemm_tile_coords(tiles_m, tiles_n, tm, tn);
  const int m0 = tm * GF_M, n0 = tn * GF_N;
  const int tid = threadIdx.x, tx = tid & 31, ty = tid >> 5;
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  const float* a_src = A + (long)min(m0 + lr, M - 1) * lda + lk;
  const float* w_src = W + (long)min(n0 + lr, N - 1) * ldw + lk;
  float acc[8][2];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i][0] = acc[i][1] = 0.f;
  for (int k0 = 0; k0 < K; k0 += GF_K) {
    const f32x4 a4 = *(const f32x4*)(a_src + k0);
    const f32x4 w4 = *(const f32x4*)(w_src + k0);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      As[lk + j][lr] = a4[j];
      Ws[lk + j][lr] = w4[j];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < GF_K; ++k) {
      const float b0 = Ws[k][tx], b1 = Ws[k][tx + 32];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float a = As[k][ty * 8 + i];
        acc[i][0] = fmaf(a, b0, acc[i][0]);
        acc[i][1] = fmaf(a, b1, acc[i][1]);
      }
    }
    __syncthreads();
  }
  const int col = n0 + tx;
  if (col < N) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int row = m0 + ty * 8 + i;
      if (row < M) epi(row, col, acc[i][0], acc[i][1]);
    }
  }
}

}  // namespace alr
