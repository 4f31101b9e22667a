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
    const float alpha = exp2f(m - m_new);
    const float p = (j < n_total) ? exp2f(sc - m_new) : 0.f;
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
// one's accumulators: in k-step ks (16 keys) lane half h supplies keys
// {4h..4h+3, 8+4h..8+4h+3} (+16 ks), and V^T is read from LDS in the same key
// order, which leaves the sum unchanged.
//
// A workgroup has 4 waves; wave w owns 32 query rows.  Key tiles of 64 keys
// are staged in LDS: K as [key][hd] rows, V transposed as [hd][key].

constexpr int AT_KT = 64;

template <int HD>
struct AttnSmem {
  static constexpr int KP = HD + 8;      // K row pitch (bf16)
  static constexpr int VP = AT_KT + 8;   // V^T row pitch (bf16)
  bf16 k[AT_KT * KP];
  bf16 vt[HD * VP];
};

// Cooperative load of one K/V tile (keys key0 .. key0+63 of rows base_row+key,
// clamped to max_row) into LDS.
template <int HD>
__device__ __forceinline__ void attn_load_tile(AttnSmem<HD>& sm, const bf16* __restrict__ Kc,
                                               const bf16* __restrict__ Vc, long kv_rs, int kvh,
                                               long base_row, int key0, int max_key) {
  constexpr int CH = AT_KT * HD / 8;  // 16-byte chunks
  for (int ch = threadIdx.x; ch < CH; ch += 256) {
    const int key = ch / (HD / 8), d8 = (ch % (HD / 8)) * 8;
    const long r = base_row + min(key0 + key, max_key);
    const u32x4 kv = *(const u32x4*)(Kc + r * kv_rs + (long)kvh * HD + d8);
    *(u32x4*)(sm.k + key * AttnSmem<HD>::KP + d8) = kv;
    const u32x4 vv = *(const u32x4*)(Vc + r * kv_rs + (long)kvh * HD + d8);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      sm.vt[(d8 + 2 * e) * AttnSmem<HD>::VP + key] = (bf16)(vv[e] & 0xFFFFu);
      sm.vt[(d8 + 2 * e + 1) * AttnSmem<HD>::VP + key] = (bf16)(vv[e] >> 16);
    }
  }
}

// One 64-key tile of the online softmax for the wave's 32 queries.
//   qb[ks]: Q^T operand (lane: query lane&31, dims 8*(lane>>5) + 16 ks .. +7)
//   key_abs0: absolute key index of tile key 0; keys with index > lim are masked.
template <int HD>
__device__ __forceinline__ void attn_tile_update(const AttnSmem<HD>& sm, const bf16x8* qb,
                                                 f32x16* o, float& m, float& l, int key_abs0,
                                                 int lim, float scale_log2) {
  const int lane = threadIdx.x & 63, h = lane >> 5, lr = lane & 31;
  f32x16 s[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
    for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks) {
      const bf16x8 a =
          as_bf16x8(*(const u32x4*)(sm.k + (kb * 32 + lr) * AttnSmem<HD>::KP + ks * 16 + h * 8));
      s[kb] = mfma32x32x16(a, qb[ks], s[kb]);
    }
  }
  float tmax = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = key_abs0 + kb * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
      const float v = (key <= lim) ? s[kb][r] * scale_log2 : -INFINITY;
      s[kb][r] = v;
      tmax = fmaxf(tmax, v);
    }
  tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
  const float m_new = fmaxf(m, tmax);
  const float mref = (m_new == -INFINITY) ? 0.f : m_new;
  const float alpha = exp2f(m - mref);
  float psum = 0.f;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float p = exp2f(s[kb][r] - mref);
      s[kb][r] = p;
      psum += p;
    }
  psum += __shfl_xor(psum, 32);
  l = l * alpha + psum;
  m = m_new;
#pragma unroll
  for (int db = 0; db < HD / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      u32x4 pw;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        pw[e] = pack2bf(s[kb][k2 * 8 + 2 * e], s[kb][k2 * 8 + 2 * e + 1]);
      const bf16x8 pb = as_bf16x8(pw);
      const int key_lo = kb * 32 + k2 * 16 + 4 * h;
#pragma unroll
      for (int db = 0; db < HD / 32; ++db) {
        const bf16* vrow = sm.vt + (db * 32 + lr) * AttnSmem<HD>::VP;
        const u32x2 v0 = *(const u32x2*)(vrow + key_lo);
        const u32x2 v1 = *(const u32x2*)(vrow + key_lo + 8);
        u32x4 va;
        va[0] = v0[0];
        va[1] = v0[1];
        va[2] = v1[0];
        va[3] = v1[1];
        o[db] = mfma32x32x16(as_bf16x8(va), pb, o[db]);
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

// Prefill work item: (seq_start_row, seq_len, kv head, first item) where items
// enumerate (query block of 32, head within the group) pairs, query-block major.
struct PrefillItem {
  int start, len, kvh, item0;
};

template <int HD>
__global__ __launch_bounds__(256) void attn_prefill_mfma_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ Kc, const bf16* __restrict__ Vc,
    bf16* __restrict__ O, const PrefillItem* __restrict__ work, AttnGeom g) {
  __shared__ AttnSmem<HD> sm;
  const PrefillItem w = work[blockIdx.x];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, h = lane >> 5, lr = lane & 31;
  const int rep = g.H / g.G;
  const int n_items = ((w.len + 31) / 32) * rep;
  const int item = w.item0 + wave;
  const bool active = item < n_items;
  const int qb = active ? item / rep : 0;
  const int head = w.kvh * rep + (active ? item % rep : 0);
  // last key needed by the workgroup: its largest query block
  const int last_item = min(w.item0 + 3, n_items - 1);
  const int wg_last_q = min(((last_item / rep) + 1) * 32, w.len) - 1;
  const int q_pos = qb * 32 + lr;            // this lane's query position
  const int q_row = min(q_pos, w.len - 1);   // clamped row for loads
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
  for (int k0 = 0; k0 <= wg_last_q; k0 += AT_KT) {
    attn_load_tile<HD>(sm, Kc, Vc, kv_rs, w.kvh, w.start, k0, w.len - 1);
    __syncthreads();
    if (active && k0 <= wave_last_q)
      attn_tile_update<HD>(sm, qbv, o, m, l, k0, q_pos, g.scale_log2);
    __syncthreads();
  }
  if (active && q_pos < w.len)
    attn_store<HD>(o, l, O + (long)(w.start + q_pos) * g.H * HD + (long)head * HD);
}

// Decode work item: a group of up to 128/rep consecutive sorted anchors of one
// sequence and one kv head.
struct DecodeItem {
  int first, count, kvh, seq_start;
};

template <int HD>
__global__ __launch_bounds__(256) void attn_decode_mfma_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ Kc, const bf16* __restrict__ Vc,
    const bf16* __restrict__ Kp, const bf16* __restrict__ Vp, long priv_rs, int n_priv,
    const int* __restrict__ apos, bf16* __restrict__ O, const DecodeItem* __restrict__ work,
    AttnGeom g) {
  __shared__ AttnSmem<HD> sm;
  const DecodeItem w = work[blockIdx.x];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, h = lane >> 5, lr = lane & 31;
  const int rep = g.H / g.G;
  const int rho = wave * 32 + lr;  // row within the group: anchor-major
  const int a_loc = rho / rep;
  const bool active = a_loc < w.count;
  const int arow = w.first + (active ? a_loc : 0);  // sorted anchor row
  const int head = w.kvh * rep + rho % rep;
  const int lim = active ? apos[arow] : -1;
  const int a_max = apos[w.first + w.count - 1];  // sorted: last is largest
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
  // rows of this wave that are active: skip tiles beyond the wave's own max anchor
  int wave_lim = lim;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) wave_lim = max(wave_lim, __shfl_xor(wave_lim, off));
  for (int k0 = 0; k0 <= a_max; k0 += AT_KT) {
    attn_load_tile<HD>(sm, Kc, Vc, kv_rs, w.kvh, w.seq_start, k0, a_max);
    __syncthreads();
    if (k0 <= wave_lim) attn_tile_update<HD>(sm, qbv, o, m, l, k0, lim, g.scale_log2);
    __syncthreads();
  }
  if (!active) return;
  // private keys of slots 1..n_priv, in chunks of 16 under the same online
  // softmax; lane half h holds q dims {8h + 16 ks + e}, the partner the rest.
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
        sc[j] = dot * g.scale_log2;
        pmax = fmaxf(pmax, sc[j]);
      }
    }
    const float m_new = fmaxf(m, pmax);
    const float alpha = exp2f(m - m_new);
#pragma unroll
    for (int db = 0; db < HD / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
    float psum = 0.f;
    for (int j = 0; j < cn; ++j) {
      const float p = exp2f(sc[j] - m_new);
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
  attn_store<HD>(o, l, O + (long)arow * g.H * HD + (long)head * HD);
}

}  // namespace alr
