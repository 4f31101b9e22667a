// Attention kernels (gfx950).
//
// Key/value layout: the shared corpus cache of one layer is [token][G][hd]
// (tokens of all sequences concatenated); the private rollout buffer of one
// layer is [anchor][slot][G][hd].  Queries and outputs are [row][H][hd].
//
// Prefill: causal attention of every corpus position over its own sequence.
// Decode: the query of (sorted) anchor r at rollout step s attends, under one
// softmax, to the shared keys of its sequence at positions 0..a_r and to its
// own private keys of slots 1..s (App. A, "Rollout implementation").
#pragma once

#include "device_common.hpp"

namespace alr {

struct AttnGeom {
  int H, G, hd;
  float scale_log2;  // log2(e) / sqrt(hd)
};

// ------------------------------------------------------------------ generic kernel
// One wave per (query row, head); lanes over keys for the scores, lanes over
// dimensions for the weighted sum.  Handles any even hd <= 256.  Used for the
// fp32 path and for head sizes the MFMA kernels do not cover.
//   prefill (priv == nullptr): row r is corpus token r, sequence start
//     row_start[r]; it sees shared rows row_start[r] .. r.
//   decode: row r is sorted anchor r with shared rows tok0[r] .. tok0[r] +
//     apos[r] where tok0[r] is its sequence start, then n_priv private slots.
template <typename T>
__global__ __launch_bounds__(256) void attn_generic_kernel(
    const T* __restrict__ Q, const T* __restrict__ Kc, const T* __restrict__ Vc,
    const T* __restrict__ Kp, const T* __restrict__ Vp, long priv_rs, int n_priv,
    const int* __restrict__ row_start, const int* __restrict__ apos, T* __restrict__ O,
    int n_rows, AttnGeom g) {
  __shared__ float qs[4][256];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const long item_raw = (long)blockIdx.x * 4 + wave;
  const bool valid = item_raw < (long)n_rows * g.H;
  const long item = valid ? item_raw : 0;
  const int row = (int)(item / g.H), head = (int)(item % g.H);
  const int kvh = head / (g.H / g.G);
  const int hd = g.hd;
  const long kv_rs = (long)g.G * hd;
  const T* q = Q + (long)row * g.H * hd + (long)head * hd;
  for (int d = lane; d < hd; d += 64) qs[wave][d] = Elt<T>::ld(q + d);
  __syncthreads();
  if (!valid) return;
  int first, n_shared, n_total;
  if (Kp == nullptr) {
    first = row_start[row];
    n_shared = row - first + 1;
    n_total = n_shared;
  } else {
    first = row_start[row];
    n_shared = apos[row] + 1;
    n_total = n_shared + n_priv;
  }
  float m = -INFINITY, l = 0.f;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int j0 = 0; j0 < n_total; j0 += 64) {
    const int j = j0 + lane;
    float sc = -INFINITY;
    if (j < n_total) {
      const T* kp = (j < n_shared) ? Kc + (long)(first + j) * kv_rs + (long)kvh * hd
                                   : Kp + (long)row * priv_rs + (long)(j - n_shared) * kv_rs +
                                         (long)kvh * hd;
      float dot = 0.f;
      for (int d = 0; d < hd; ++d) dot = fmaf(qs[wave][d], Elt<T>::ld(kp + d), dot);
      sc = dot * g.scale_log2;
    }
    const float m_new = fmaxf(m, wave_max(sc));
    const float alpha = fast_exp2(m - m_new);
    const float p = (j < n_total) ? fast_exp2(sc - m_new) : 0.f;
    l = l * alpha + wave_sum(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] *= alpha;
    const int cnt = min(64, n_total - j0);
    for (int jj = 0; jj < cnt; ++jj) {
      const float pj = __shfl(p, jj);
      const int jk = j0 + jj;
      const T* vp = (jk < n_shared) ? Vc + (long)(first + jk) * kv_rs + (long)kvh * hd
                                    : Vp + (long)row * priv_rs + (long)(jk - n_shared) * kv_rs +
                                          (long)kvh * hd;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = lane + 64 * i;
        if (d < hd) acc[i] = fmaf(pj, Elt<T>::ld(vp + d), acc[i]);
      }
    }
    m = m_new;
  }
  T* o = O + (long)row * g.H * hd + (long)head * hd;
  const float inv = 1.f / l;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int d = lane + 64 * i;
    if (d < hd) Elt<T>::st(o + d, acc[i] * inv);
  }
}

// ------------------------------------------------------------------ MFMA kernels (bf16)
//
// Both compute S^T = K Q^T with 32x32x16 MFMAs, so that a lane owns one query
// (column) and 16 keys (rows): the per-query softmax statistics need only a
// lane-local reduction plus one exchange with lane ^ 32.  O^T = V^T P^T then
// keeps the same column-per-query layout, so rescaling by the running max is
// lane-local too.  P^T is fed to the second MFMA straight from the first
// one's accumulators: in a 16-key k-step lane half h supplies keys
// {4h..4h+3, 8+4h..8+4h+3}; the V^T tile keeps its keys in that order inside
// each 16-key group, so each V^T operand is one 16-byte LDS read.
//
// The shared V cache is stored transposed, [G][hd][column] per layer, with
// every sequence's columns starting at a multiple of 64, so a 64-key V^T tile
// is 16-byte loads of contiguous keys.  K tiles are [key][hd].  Both tiles are
// XOR-swizzled in 16-byte chunks so the MFMA operand reads are free of LDS
// bank conflicts.  Tiles are double-buffered: the next tile's global loads are
// in flight while the current one is consumed.

constexpr int AT_KT = 64;
constexpr int AT_DECODE_CHUNK = 512;  // keys per decode work item

template <int NCH>
__device__ __forceinline__ int chunk_swz(int r, int c) {
  if constexpr (NCH == 16)
    return c ^ (r & 15);
  else
    return c ^ ((r & 7) ^ ((r >> 3) & 1));
}

template <int HD>
struct AttnTile {
  bf16 k[AT_KT * HD];   // [key][dim]
  bf16 vt[HD * AT_KT];  // [dim][key]
};

template <int HD>
struct AttnStage {
  u32x4 k[HD / 32];
  u32x4 v[HD / 32];
};

// Global loads of one tile: keys k0..k0+63 of a sequence whose key 0 is token
// row krow0 of the K cache and column vcol0 of the V^T cache.  Keys beyond
// max_key read a clamped K row and zeros for V (they are masked anyway; the
// zeros keep unwritten padding out of the sums).
template <int HD>
__device__ __forceinline__ void attn_gload(AttnStage<HD>& st, const bf16* __restrict__ Kc,
                                           long kv_rs, int kvh, long krow0,
                                           const bf16* __restrict__ vT, long vt_stride,
                                           long vcol0, int k0, int max_key) {
  constexpr int NCHK = HD / 8;
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < HD / 32; ++i) {
    const int ch = tid + 256 * i, key = ch / NCHK, c = ch % NCHK;
    st.k[i] = *(const u32x4*)(Kc + (krow0 + min(k0 + key, max_key)) * kv_rs + (long)kvh * HD + c * 8);
  }
#pragma unroll
  for (int i = 0; i < HD / 32; ++i) {
    const int ch = tid + 256 * i, dim = ch >> 3, c = ch & 7;
    const int kf = k0 + c * 8;
    u32x4 v = *(const u32x4*)(vT + (long)(kvh * HD + dim) * vt_stride + vcol0 + kf);
    if (kf + 7 > max_key) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int ka = kf + 2 * e;
        uint32_t w = v[e];
        if (ka > max_key) w &= 0xFFFF0000u;
        if (ka + 1 > max_key) w &= 0x0000FFFFu;
        v[e] = w;
      }
    }
    st.v[i] = v;
  }
}

template <int HD>
__device__ __forceinline__ void attn_lstore(const AttnStage<HD>& st, AttnTile<HD>& t) {
  constexpr int NCHK = HD / 8;
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < HD / 32; ++i) {
    const int ch = tid + 256 * i, key = ch / NCHK, c = ch % NCHK;
    *(u32x4*)(t.k + key * HD + chunk_swz<NCHK>(key, c) * 8) = st.k[i];
  }
#pragma unroll
  for (int i = 0; i < HD / 32; ++i) {
    const int ch = tid + 256 * i, dim = ch >> 3, c = ch & 7;
    const int g = c >> 1, q = c & 1;  // 16-key group, which half of it
    // keys 8c..8c+3 -> chunk 2g (half q); keys 8c+4..8c+7 -> chunk 2g+1 (half q)
    u32x2 lo, hi;
    lo[0] = st.v[i][0];
    lo[1] = st.v[i][1];
    hi[0] = st.v[i][2];
    hi[1] = st.v[i][3];
    *(u32x2*)(t.vt + dim * AT_KT + chunk_swz<8>(dim, 2 * g) * 8 + q * 4) = lo;
    *(u32x2*)(t.vt + dim * AT_KT + chunk_swz<8>(dim, 2 * g + 1) * 8 + q * 4) = hi;
  }
}

// One 64-key tile of the online softmax for the wave's 32 queries.
//   qb[ks]: Q^T operand (lane: query lane&31, dims 8*(lane>>5) + 16 ks .. +7)
//   key_abs0: key index of tile key 0; with MASK, keys with index > lim are
//   masked (tiles entirely at or below every lane's lim skip the masking).
//   m is the running max of the raw scores; scale_log2 = log2(e)/sqrt(hd) is
//   applied inside the exponent.
template <int HD, bool MASK>
__device__ __forceinline__ void attn_tile_update(const AttnTile<HD>& t, const bf16x8* qb,
                                                 f32x16* o, float& m, float& l, int key_abs0,
                                                 int lim, float scale_log2) {
  constexpr int NCHK = HD / 8;
  const int lane = threadIdx.x & 63, h = lane >> 5, lr = lane & 31;
  f32x16 s[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
    for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
    const int key = kb * 32 + lr;
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks) {
      const bf16x8 a =
          as_bf16x8(*(const u32x4*)(t.k + key * HD + chunk_swz<NCHK>(key, 2 * ks + h) * 8));
      s[kb] = mfma32x32x16(a, qb[ks], s[kb]);
    }
  }
  float tmax = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      if constexpr (MASK) {
        const int key = key_abs0 + kb * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (key > lim) s[kb][r] = -INFINITY;
      }
      tmax = fmaxf(tmax, s[kb][r]);
    }
  tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
  const float m_new = fmaxf(m, tmax);
  const float mref = (m_new == -INFINITY) ? 0.f : m_new * scale_log2;
  const bool grew = m_new > m;
  const float alpha = grew ? fast_exp2(m * scale_log2 - mref) : 1.f;
  float psum = 0.f;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float p = fast_exp2(fmaf(s[kb][r], scale_log2, -mref));
      s[kb][r] = p;
      psum += p;
    }
  psum += __shfl_xor(psum, 32);
  l = l * alpha + psum;
  m = m_new;
  if (__any(grew)) {
#pragma unroll
    for (int db = 0; db < HD / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
  }
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      u32x4 pw;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        pw[e] = pack2bf(s[kb][k2 * 8 + 2 * e], s[kb][k2 * 8 + 2 * e + 1]);
      const bf16x8 pb = as_bf16x8(pw);
      const int c = 2 * (kb * 2 + k2) + h;
#pragma unroll
      for (int db = 0; db < HD / 32; ++db) {
        const int dim = db * 32 + lr;
        const bf16x8 va = as_bf16x8(*(const u32x4*)(t.vt + dim * AT_KT + chunk_swz<8>(dim, c) * 8));
        o[db] = mfma32x32x16(va, pb, o[db]);
      }
    }
}

// Store O^T / l for the lane's query into out (row pointer, natural order).
template <int HD>
__device__ __forceinline__ void attn_store(const f32x16* o, float l, bf16* out_row) {
  const int lane = threadIdx.x & 63, h = lane >> 5;
  const float inv = 1.f / l;
#pragma unroll
  for (int db = 0; db < HD / 32; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int d = db * 32 + 8 * i + 4 * h;
      u32x2 w;
      w[0] = pack2bf(o[db][4 * i] * inv, o[db][4 * i + 1] * inv);
      w[1] = pack2bf(o[db][4 * i + 2] * inv, o[db][4 * i + 3] * inv);
      *(u32x2*)(out_row + d) = w;
    }
}

// Prefill work item: (first K-cache row of the sequence, its first V^T
// column, length, kv head, first item) where items enumerate (query block of
// 32, head within the group) pairs, query-block major.
struct PrefillItem {
  int start, vcol, len, kvh, item0;
};

template <int HD>
__global__ __launch_bounds__(256, 2) void attn_prefill_mfma_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ Kc, const bf16* __restrict__ vT,
    long vt_stride, bf16* __restrict__ O, const PrefillItem* __restrict__ work, AttnGeom g) {
  __shared__ AttnTile<HD> tiles[2];
  const PrefillItem w = work[blockIdx.x];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, h = lane >> 5, lr = lane & 31;
  const int rep = g.H / g.G;
  const int n_items = ((w.len + 31) / 32) * rep;
  const int item = w.item0 + wave;
  const bool active = item < n_items;
  const int qb = active ? item / rep : 0;
  const int head = w.kvh * rep + (active ? item % rep : 0);
  const int last_item = min(w.item0 + 3, n_items - 1);
  const int wg_last_q = min(((last_item / rep) + 1) * 32, w.len) - 1;
  const int q_pos = qb * 32 + lr;
  const int q_row = min(q_pos, w.len - 1);
  const long kv_rs = (long)g.G * HD;
  bf16x8 qbv[HD / 16];
  {
    const bf16* qp = Q + (long)(w.start + q_row) * g.H * HD + (long)head * HD + h * 8;
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks) qbv[ks] = as_bf16x8(*(const u32x4*)(qp + ks * 16));
  }
  f32x16 o[HD / 32];
#pragma unroll
  for (int db = 0; db < HD / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  float m = -INFINITY, l = 0.f;
  const int wave_last_q = min(qb * 32 + 31, w.len - 1);
  const int nt = wg_last_q / AT_KT + 1;
  AttnStage<HD> st;
  attn_gload<HD>(st, Kc, kv_rs, w.kvh, w.start, vT, vt_stride, w.vcol, 0, w.len - 1);
  attn_lstore<HD>(st, tiles[0]);
  __syncthreads();
  for (int it = 0; it < nt; ++it) {
    const int k0 = it * AT_KT;
    if (it + 1 < nt)
      attn_gload<HD>(st, Kc, kv_rs, w.kvh, w.start, vT, vt_stride, w.vcol, k0 + AT_KT, w.len - 1);
    if (active && k0 <= wave_last_q) {
      if (k0 + AT_KT - 1 > qb * 32)  // some key of the tile lies beyond some query: mask
        attn_tile_update<HD, true>(tiles[it & 1], qbv, o, m, l, k0, q_pos, g.scale_log2);
      else
        attn_tile_update<HD, false>(tiles[it & 1], qbv, o, m, l, k0, q_pos, g.scale_log2);
    }
    if (it + 1 < nt) attn_lstore<HD>(st, tiles[(it + 1) & 1]);
    __syncthreads();
  }
  if (active && q_pos < w.len)
    attn_store<HD>(o, l, O + (long)(w.start + q_pos) * g.H * HD + (long)head * HD);
}

// Decode work item: a group of up to 128/rep consecutive sorted anchors of one
// sequence, one kv head, and the shared keys [kbeg, kend) of that sequence.
// The item writes, per row (anchor-major, then head within the group), the
// partial softmax state: running max m and sum l (log2 domain) and the
// unnormalised output; attn_decode_combine_kernel merges the items of a group
// (the item holding the final chunk also folds in the anchor's private keys).
struct DecodeItem {
  int first, count, kvh, krow0, vcol0, kbeg, kend, part, last;  // last: final chunk of the group
};

template <int HD>
__global__ __launch_bounds__(256, 2) void attn_decode_mfma_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ Kc, const bf16* __restrict__ vT,
    long vt_stride, const bf16* __restrict__ Kp, const bf16* __restrict__ Vp, long priv_rs,
    int n_priv, const int* __restrict__ apos, const DecodeItem* __restrict__ work,
    float* __restrict__ part_o, float* __restrict__ part_ml, AttnGeom g) {
  __shared__ AttnTile<HD> tiles[2];
  const DecodeItem w = work[blockIdx.x];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, h = lane >> 5, lr = lane & 31;
  const int rep = g.H / g.G;
  const int rho = wave * 32 + lr;  // row within the group: anchor-major
  const int a_loc = rho / rep;
  const bool active = a_loc < w.count;
  const int arow = w.first + (active ? a_loc : 0);
  const int head = w.kvh * rep + rho % rep;
  const int lim = active ? min(apos[arow], w.kend - 1) : -1;
  const long kv_rs = (long)g.G * HD;
  bf16x8 qbv[HD / 16];
  {
    const bf16* qp = Q + (long)arow * g.H * HD + (long)head * HD + h * 8;
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks) qbv[ks] = as_bf16x8(*(const u32x4*)(qp + ks * 16));
  }
  f32x16 o[HD / 32];
#pragma unroll
  for (int db = 0; db < HD / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  float m = -INFINITY, l = 0.f;
  int wave_lim = lim, wave_min = active ? lim : 0x7FFFFFFF;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    wave_lim = max(wave_lim, __shfl_xor(wave_lim, off));
    wave_min = min(wave_min, __shfl_xor(wave_min, off));
  }
  const int nt = (w.kend - w.kbeg + AT_KT - 1) / AT_KT;
  AttnStage<HD> st;
  attn_gload<HD>(st, Kc, kv_rs, w.kvh, w.krow0, vT, vt_stride, w.vcol0, w.kbeg, w.kend - 1);
  attn_lstore<HD>(st, tiles[0]);
  __syncthreads();
  for (int it = 0; it < nt; ++it) {
    const int k0 = w.kbeg + it * AT_KT;
    if (it + 1 < nt)
      attn_gload<HD>(st, Kc, kv_rs, w.kvh, w.krow0, vT, vt_stride, w.vcol0, k0 + AT_KT,
                     w.kend - 1);
    if (k0 <= wave_lim) {
      if (k0 + AT_KT - 1 > wave_min)
        attn_tile_update<HD, true>(tiles[it & 1], qbv, o, m, l, k0, lim, g.scale_log2);
      else
        attn_tile_update<HD, false>(tiles[it & 1], qbv, o, m, l, k0, lim, g.scale_log2);
    }
    if (it + 1 < nt) attn_lstore<HD>(st, tiles[(it + 1) & 1]);
    __syncthreads();
  }
  if (!active) return;
  if (w.last) {
    // the anchor's private keys of slots 1..n_priv join the last chunk's softmax;
    // lane half h holds q dims {8h + 16 ks + e}, the partner lane the rest
    const bf16* kp = Kp + (long)arow * priv_rs + (long)w.kvh * HD;
    const bf16* vp = Vp + (long)arow * priv_rs + (long)w.kvh * HD;
    for (int c0 = 0; c0 < n_priv; c0 += 16) {
      const int cn = min(16, n_priv - c0);
      float sc[16];
      float pmax = -INFINITY;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        sc[j] = -INFINITY;
        if (j < cn) {
          float dot = 0.f;
#pragma unroll
          for (int ks = 0; ks < HD / 16; ++ks) {
            const u32x4 kw = *(const u32x4*)(kp + (long)(c0 + j) * kv_rs + ks * 16 + h * 8);
            const u32x4 qw = __builtin_bit_cast(u32x4, qbv[ks]);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              dot = fmaf(bf2f((bf16)(qw[e] & 0xFFFFu)), bf2f((bf16)(kw[e] & 0xFFFFu)), dot);
              dot = fmaf(bf2f((bf16)(qw[e] >> 16)), bf2f((bf16)(kw[e] >> 16)), dot);
            }
          }
          dot += __shfl_xor(dot, 32);
          sc[j] = dot;  // raw score, like m
          pmax = fmaxf(pmax, sc[j]);
        }
      }
      const float m_new = fmaxf(m, pmax);
      const float mref = m_new * g.scale_log2;
      const float alpha = fast_exp2(m * g.scale_log2 - mref);
#pragma unroll
      for (int db = 0; db < HD / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
      float psum = 0.f;
      for (int j = 0; j < cn; ++j) {
        const float p = fast_exp2(fmaf(sc[j], g.scale_log2, -mref));
        psum += p;
        const bf16* vj = vp + (long)(c0 + j) * kv_rs;
#pragma unroll
        for (int db = 0; db < HD / 32; ++db)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const u32x2 vv = *(const u32x2*)(vj + db * 32 + 8 * i + 4 * h);
            o[db][4 * i] = fmaf(p, bf2f((bf16)(vv[0] & 0xFFFFu)), o[db][4 * i]);
            o[db][4 * i + 1] = fmaf(p, bf2f((bf16)(vv[0] >> 16)), o[db][4 * i + 1]);
            o[db][4 * i + 2] = fmaf(p, bf2f((bf16)(vv[1] & 0xFFFFu)), o[db][4 * i + 2]);
            o[db][4 * i + 3] = fmaf(p, bf2f((bf16)(vv[1] >> 16)), o[db][4 * i + 3]);
          }
      }
      l = l * alpha + psum;
      m = m_new;
    }
  }
  const long prow = (long)w.part * 128 + rho;
  float* po = part_o + prow * HD;
#pragma unroll
  for (int db = 0; db < HD / 32; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f32x4 v;
      v[0] = o[db][4 * i];
      v[1] = o[db][4 * i + 1];
      v[2] = o[db][4 * i + 2];
      v[3] = o[db][4 * i + 3];
      *(f32x4*)(po + db * 32 + 8 * i + 4 * h) = v;
    }
  if (h == 0) {
    part_ml[prow * 2] = m * g.scale_log2;  // log2 domain for the combine
    part_ml[prow * 2 + 1] = l;
  }
}

// Group of sorted anchors as the combine kernel sees it.
struct DecodeGroup {
  int first, nchunk, part0;  // part index of (kv head 0, chunk 0); kv head g adds g*nchunk
};

// One wave per (sorted anchor r, query head j): merge the chunk partials of
// its group (log2-domain max m, sum l, unnormalised output) into the
// attention output.  Lanes own dims lane + 64 e; the loads of different
// chunks are independent, so they are issued together.
template <int HD>
__global__ __launch_bounds__(256) void attn_decode_combine_kernel(
    const int* __restrict__ grp_of_row, const DecodeGroup* __restrict__ groups,
    const float* __restrict__ part_o, const float* __restrict__ part_ml, bf16* __restrict__ O,
    int n_rows, AttnGeom g) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const long item = (long)blockIdx.x * 4 + wave;
  if (item >= (long)n_rows * g.H) return;  // no barrier in this kernel
  const int r = (int)(item / g.H), j = (int)(item % g.H);
  const int rep = g.H / g.G, kvh = j / rep;
  const DecodeGroup grp = groups[grp_of_row[r]];
  const int rho = (r - grp.first) * rep + j % rep;
  constexpr int DPL = HD / 64;  // dims per lane
  const long p0 = (long)(grp.part0 + kvh * grp.nchunk) * 128 + rho;  // chunk c adds c*128
  // chunk maxima: lane c reads chunk c's m (nchunk <= 64 per pass)
  float mtot = -INFINITY;
  for (int c0 = 0; c0 < grp.nchunk; c0 += 64) {
    const int c = c0 + lane;
    const float mc = (c < grp.nchunk) ? part_ml[(p0 + (long)c * 128) * 2] : -INFINITY;
    mtot = fmaxf(mtot, wave_max(mc));
  }
  float ltot = 0.f, acc[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) acc[e] = 0.f;
#pragma unroll 4
  for (int c = 0; c < grp.nchunk; ++c) {
    const long prow = p0 + (long)c * 128;
    const float mc = part_ml[prow * 2];
    const float a = (mc == -INFINITY) ? 0.f : fast_exp2(mc - mtot);
    ltot = fmaf(part_ml[prow * 2 + 1], a, ltot);
#pragma unroll
    for (int e = 0; e < DPL; ++e) acc[e] = fmaf(part_o[prow * HD + lane + 64 * e], a, acc[e]);
  }
  const float inv = 1.f / ltot;
  bf16* out = O + (long)r * g.H * HD + (long)j * HD;
#pragma unroll
  for (int e = 0; e < DPL; ++e) out[lane + 64 * e] = f2bf(acc[e] * inv);
}

}  // namespace alr
