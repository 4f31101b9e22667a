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
// every sequence's columns starting at a multiple of 64 and each aligned group
// of 16 keys already in that lane-half order (vt_perm), so a 64-key V^T tile is
// copied as contiguous 16-byte chunks.  K tiles are [key][hd].  Both tiles are
// XOR-swizzled in 16-byte chunks so the MFMA operand reads are free of LDS
// bank conflicts.  Tiles go from global memory straight into LDS
// (AttnCopier) and are double-buffered: the next tile's copies are in
// flight while the current one is consumed.

constexpr int AT_KT = 64;
// Decode split: the shared keys of every (anchor group, kv head) are cut into
// chunks of a common number ct of 64-key tiles.  The host picks ct to
// minimise the simulated makespan (list scheduling, largest item first, two
// workgroups per CU, an item costing its tiles + AT_DECODE_ITEM_OVERHEAD)
// among the ct that give at most AT_DECODE_MAX_ITEMS items and never fewer
// than AT_DECODE_MIN_TILES tiles per item.
constexpr int AT_DECODE_MAX_ITEMS = 2048;
constexpr int AT_DECODE_ITEM_OVERHEAD = 3;  // prologue, partial store and merge, in tiles
constexpr int AT_DECODE_MIN_TILES = 4;

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

__device__ __forceinline__ uint32_t lds_byte_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// One wave-wide 1 KB copy global -> LDS (global_load_lds_dwordx4): lane i
// fetches 16 bytes at gbase + voff and writes them to LDS byte m0 + 16 i.  No
// VGPR holds the data and no ds_write is issued.  The compiler does not see the
// copy, so every wait on it is explicit (attn_wait_copies).
// m0 is named as clobbered for the reader; the compiler reserves it and uses
// it in these kernels only for such copies (checked in their assembly).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void copy_1k(uint32_t m0, uint32_t voff, const void* gbase) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
               :
               : "s"(m0), "v"(voff), "s"(gbase)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// s_waitcnt vmcnt(0) with the other counters left alone: this wave's copies
// (and any earlier global loads) have landed.
__device__ __forceinline__ void attn_wait_copies() {
  __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));
}

// Makes the loads of v complete here: the compiler waits for them before this
// point.  The tile copies are invisible to its wait counting, so a load left
// outstanding into the loop would make its first use there wait for every
// copy issued since as well (vmcnt counts both, in issue order).
template <int N>
__device__ __forceinline__ void attn_hold_loaded(const u32x4 (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : : "v"(v[i]));
}

// Copies of 64-key tiles into LDS by the workgroup's 4 waves, for keys k0..k0+63
// of a sequence whose key 0 is token row krow0 of the K cache and column vcol0
// of the V^T cache.  Keys beyond max_key fetch K row max_key (they are masked
// anyway); the V^T cache already holds its keys in the value MFMA's order
// (vt_perm) and zeros in the columns that pad a sequence to a multiple of 64.
// Each operand is HD/8 wave-wide 1 KB copies; copy j*4 + w belongs to wave w,
// and lane l of it fills LDS chunk p = (j*4 + w)*64 + l of the operand's
// XOR-swizzled layout, i.e. it fetches the global chunk the swizzle maps there.
// The lane's part of each offset is formed once per work item; a tile adds
// its first key (a row multiple for K, a column for V^T).  Byte offsets from
// the layer's cache base fit 32 bits (checked on the host).
template <int HD>
struct AttnCopier {
  static constexpr int NCHK = HD / 8;
  static constexpr int NX = HD / 32;  // copies per wave per operand
  uint32_t koff[NX], voff[NX];        // byte offsets of the lane's chunks at k0 = 0
  int key[NX];                        // the lane's key within the tile, per K copy
  uint32_t krow_bytes;                // bytes of one K-cache row
  int wave;

  __device__ __forceinline__ AttnCopier(long kv_rs, int kvh, long krow0, long vt_stride,
                                        long vcol0) {
    const int lane = threadIdx.x & 63;
    wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    krow_bytes = (uint32_t)(kv_rs * 2);
#pragma unroll
    for (int j = 0; j < NX; ++j) {
      const int p = (j * 4 + wave) * 64 + lane;
      key[j] = p / NCHK;
      const int ck = chunk_swz<NCHK>(key[j], p % NCHK);
      koff[j] = (uint32_t)((krow0 * kv_rs + (long)kvh * HD + ck * 8) * 2);
      const int dim = p >> 3, cv = chunk_swz<8>(dim, p & 7);
      voff[j] = (uint32_t)((((long)kvh * HD + dim) * vt_stride + vcol0 + cv * 8) * 2);
    }
  }

  __device__ __forceinline__ void tile(AttnTile<HD>& t, const bf16* __restrict__ Kc,
                                       const bf16* __restrict__ vT, int k0, int max_key) const {
    const uint32_t kb = lds_byte_addr(t.k), vb = lds_byte_addr(t.vt);
    if (k0 + AT_KT - 1 <= max_key) {  // uniform: no key of the tile past max_key
#pragma unroll
      for (int j = 0; j < NX; ++j)
        copy_1k(kb + (j * 4 + wave) * 1024, koff[j] + (uint32_t)(k0 + key[j]) * krow_bytes, Kc);
    } else {
#pragma unroll
      for (int j = 0; j < NX; ++j)
        copy_1k(kb + (j * 4 + wave) * 1024,
                koff[j] + (uint32_t)min(k0 + key[j], max_key) * krow_bytes, Kc);
    }
#pragma unroll
    for (int j = 0; j < NX; ++j)
      copy_1k(vb + (j * 4 + wave) * 1024, voff[j] + (uint32_t)k0 * 2, vT);
  }
};

// One 64-key tile of the online softmax for the wave's 32 queries.
//   qb[ks]: Q^T operand (lane: query lane&31, dims 8*(lane>>5) + 16 ks .. +7)
//   key_abs0: key index of tile key 0; with MASK, keys with index > lim are
//   masked (tiles entirely at or below every lane's lim skip the masking).
//   m is the running max of the raw scores; scale_log2 = log2(e)/sqrt(hd) is
//   applied inside the exponent.
//   EARLY_V: the tile's V^T fragments are read between the score MFMAs and the
//   softmax (64 more live registers at hd 128), so that the softmax covers their
//   LDS latency instead of each value MFMA waiting on its read.  The prefill
//   kernel takes it (3% faster); the decode kernel measured no gain from it.
template <int HD, bool MASK, bool EARLY_V = false>
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
  u32x4 vf[2][2][HD / 32];
  if constexpr (EARLY_V) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
        for (int db = 0; db < HD / 32; ++db) {
          const int dim = db * 32 + lr;
          vf[kb][k2][db] =
              *(const u32x4*)(t.vt + dim * AT_KT + chunk_swz<8>(dim, 2 * (kb * 2 + k2) + h) * 8);
        }
    // keeps the reads ahead of the softmax (the scheduler would sink them to their uses)
    __builtin_amdgcn_sched_barrier(0);
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
  tmax = max_xor32(tmax);
  // The reference m moves only when the tile's max exceeds it by more than 8
  // in the exponent (or on the first keys): the weights exp2(s - m) then stay
  // below 256 and the accumulators are rescaled on few tiles, not on every
  // tile whose max grew.  o, l and m stay consistent, so o / l is unchanged.
  const bool grew = tmax * scale_log2 > m * scale_log2 + 8.f;
  const float m_new = grew ? tmax : m;
  const float mref = (m_new == -INFINITY) ? 0.f : m_new * scale_log2;
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
  psum = sum_xor32(psum);
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
        const u32x4 va = EARLY_V ? vf[kb][k2][db]
                                 : *(const u32x4*)(t.vt + dim * AT_KT + chunk_swz<8>(dim, c) * 8);
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
    u32x4 qraw[HD / 16];
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks) qraw[ks] = *(const u32x4*)(qp + ks * 16);
    attn_hold_loaded<HD / 16>(qraw);
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks) qbv[ks] = as_bf16x8(qraw[ks]);
  }
  f32x16 o[HD / 32];
#pragma unroll
  for (int db = 0; db < HD / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  float m = -INFINITY, l = 0.f;
  const int wave_last_q = min(qb * 32 + 31, w.len - 1);
  const int nt = wg_last_q / AT_KT + 1;
  const AttnCopier<HD> cp(kv_rs, w.kvh, w.start, vt_stride, w.vcol);
  cp.tile(tiles[0], Kc, vT, 0, w.len - 1);
  attn_wait_copies();
  __syncthreads();
  for (int it = 0; it < nt; ++it) {
    const int k0 = it * AT_KT;
    // the next tile streams into the other buffer while this one is consumed
    if (it + 1 < nt) cp.tile(tiles[(it + 1) & 1], Kc, vT, k0 + AT_KT, w.len - 1);
    if (active && k0 <= wave_last_q) {
      if (k0 + AT_KT - 1 > qb * 32)  // some key of the tile lies beyond some query: mask
        attn_tile_update<HD, true, true>(tiles[it & 1], qbv, o, m, l, k0, q_pos, g.scale_log2);
      else
        attn_tile_update<HD, false, true>(tiles[it & 1], qbv, o, m, l, k0, q_pos, g.scale_log2);
    }
    attn_wait_copies();
    __syncthreads();
  }
  if (active && q_pos < w.len)
    attn_store<HD>(o, l, O + (long)(w.start + q_pos) * g.H * HD + (long)head * HD);
}

// Decode work item: a group of up to 128/rep consecutive sorted anchors of one
// sequence, one kv head, and the shared keys [kbeg, kend) of that sequence.
// The item writes, per row (anchor-major, then head within the group), the
// partial softmax state over those keys: the reference max m (log2 domain; -inf
// when none of the keys is visible to the row), the sum l of the weights, and the
// output normalised by l, in fp16.  attn_decode_combine_kernel merges the
// items of a group and adds the anchors' private rollout keys.  An item with
// count = 0 is padding and does nothing.
struct DecodeItem {
  int first, count, kvh, krow0, vcol0, kbeg, kend, part;
};

template <int HD>
__global__ __launch_bounds__(256, 2) void attn_decode_mfma_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ Kc, const bf16* __restrict__ vT,
    long vt_stride, const int* __restrict__ apos, const DecodeItem* __restrict__ work,
    uint16_t* __restrict__ part_o, float* __restrict__ part_ml, AttnGeom g) {
  __shared__ AttnTile<HD> tiles[2];
  const DecodeItem w = work[blockIdx.x];
  if (w.count == 0) return;  // uniform over the workgroup
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
    u32x4 qraw[HD / 16];
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks) qraw[ks] = *(const u32x4*)(qp + ks * 16);
    attn_hold_loaded<HD / 16>(qraw);
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks) qbv[ks] = as_bf16x8(qraw[ks]);
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
  const AttnCopier<HD> cp(kv_rs, w.kvh, w.krow0, vt_stride, w.vcol0);
  cp.tile(tiles[0], Kc, vT, w.kbeg, w.kend - 1);
  attn_wait_copies();
  __syncthreads();
  for (int it = 0; it < nt; ++it) {
    const int k0 = w.kbeg + it * AT_KT;
    if (it + 1 < nt) cp.tile(tiles[(it + 1) & 1], Kc, vT, k0 + AT_KT, w.kend - 1);
    if (k0 <= wave_lim) {
      if (k0 + AT_KT - 1 > wave_min)
        attn_tile_update<HD, true>(tiles[it & 1], qbv, o, m, l, k0, lim, g.scale_log2);
      else
        attn_tile_update<HD, false>(tiles[it & 1], qbv, o, m, l, k0, lim, g.scale_log2);
    }
    attn_wait_copies();
    __syncthreads();
  }
  if (!active) return;
  // the chunk's output normalised by its own sum, in fp16 (a convex combination
  // of value rows: no range issue), zeros when no key of the chunk is visible
  const long prow = (long)w.part * 128 + rho;
  uint16_t* po = part_o + prow * HD;
  const float inv = (l > 0.f) ? 1.f / l : 0.f;
#pragma unroll
  for (int db = 0; db < HD / 32; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      u32x2 v;
      v[0] = pack2h(o[db][4 * i] * inv, o[db][4 * i + 1] * inv);
      v[1] = pack2h(o[db][4 * i + 2] * inv, o[db][4 * i + 3] * inv);
      *(u32x2*)(po + db * 32 + 8 * i + 4 * h) = v;
    }
  if (h == 0) {
    part_ml[prow * 2] = (l > 0.f) ? m * g.scale_log2 : -INFINITY;  // log2 domain
    part_ml[prow * 2 + 1] = l;
  }
}

// Group of sorted anchors as the planner sees it (the combine kernel reads, per
// sorted row, its first partial row and the chunk count: the row table).
struct DecodeGroup {
  int first, nchunk, part0;  // part index of (kv head 0, chunk 0); kv head g adds g*nchunk
};

// One wave per (sorted anchor r, kv head): for each query head j of the kv
// head's group it merges the chunk partials of the shared keys (log2-domain
// reference m, sum l, output normalised by l in fp16) and then the anchor's private rollout
// keys 1..n_priv (one softmax over both), and writes the attention output.
// A head is handled by HD/8 lanes with 8 dimensions each, so one pass covers
// 64/(HD/8) heads and a score is a reduction over those lanes.  The private
// key and value rows of the kv head are read by every head of the pass.
template <int HD>
__global__ __launch_bounds__(256, 4) void attn_decode_combine_kernel(
    const int2* __restrict__ rowinfo,
    const uint16_t* __restrict__ part_o, const float* __restrict__ part_ml,
    const bf16* __restrict__ Q, const bf16* __restrict__ Kp, const bf16* __restrict__ Vp,
    long priv_rs, int n_priv, bf16* __restrict__ O, int n_rows, AttnGeom g) {
  constexpr int LPH = HD / 8;    // lanes per head
  constexpr int HPP = 64 / LPH;  // heads per pass
  constexpr int PB = 8;          // private keys per block (bounds the registers: 4 waves per SIMD)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const long item = (long)blockIdx.x * 4 + wave;
  if (item >= (long)n_rows * g.G) return;  // no barrier in this kernel
  const int r = (int)(item / g.G), kvh = (int)(item % g.G);
  const int rep = g.H / g.G;
  // (first partial row of the anchor at kv head 0 and chunk 0, chunks of its group)
  const int2 ri = rowinfo[r];
  const int nchunk = ri.y;
  const int hh = lane / LPH, dl = lane % LPH;
  const long kv_rs = (long)g.G * HD;
  const bf16* kp = Kp + (long)r * priv_rs + (long)kvh * HD + dl * 8;
  const bf16* vp = Vp + (long)r * priv_rs + (long)kvh * HD + dl * 8;
  for (int j0 = 0; j0 < rep; j0 += HPP) {
    const int jl = j0 + hh;
    const bool act = jl < rep;
    const int jc = act ? jl : 0;
    const int head = kvh * rep + jc;
    float q[8];
    {
      const u32x4 qw = *(const u32x4*)(Q + ((long)r * g.H + head) * HD + dl * 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        q[2 * e] = bf2f((bf16)(qw[e] & 0xFFFFu));
        q[2 * e + 1] = bf2f((bf16)(qw[e] >> 16));
      }
    }
    // shared keys: merge the chunk partials
    const long p0 = (long)ri.x + (long)kvh * nchunk * 128 + jc;  // chunk c adds c*128
    // one online pass: all of a round's loads are independent of each other
    float mt = -INFINITY, lt = 0.f, acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
#pragma unroll 4
    for (int c = 0; c < nchunk; ++c) {
      const long prow = p0 + (long)c * 128;
      const f32x2 ml = *(const f32x2*)(part_ml + prow * 2);
      const float mc = ml[0], lc = ml[1];
      const u32x4 ow = *(const u32x4*)(part_o + prow * HD + dl * 8);
      const float mn = fmaxf(mt, mc);
      const float alpha = (mt == -INFINITY) ? 0.f : fast_exp2(mt - mn);
      const float wgt = (mc == -INFINITY) ? 0.f : lc * fast_exp2(mc - mn);
      lt = fmaf(lt, alpha, wgt);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] = fmaf(acc[2 * e], alpha, wgt * h_lo(ow[e]));
        acc[2 * e + 1] = fmaf(acc[2 * e + 1], alpha, wgt * h_hi(ow[e]));
      }
      mt = mn;
    }
    // private keys, in blocks of PB: all key and value rows of a block are
    // loaded first (rows past n_priv re-read the last valid one), then the
    // scores, one rescale, and the weighted values
    for (int t0 = 0; t0 < n_priv; t0 += PB) {
      const int tn = min(PB, n_priv - t0);
      u32x4 kw[PB], vw[PB];
#pragma unroll
      for (int t = 0; t < PB; ++t) kw[t] = *(const u32x4*)(kp + (long)(t0 + min(t, tn - 1)) * kv_rs);
#pragma unroll
      for (int t = 0; t < PB; ++t) vw[t] = *(const u32x4*)(vp + (long)(t0 + min(t, tn - 1)) * kv_rs);
      float sc[PB];
      float bmax = -INFINITY;
#pragma unroll
      for (int t = 0; t < PB; ++t) {
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          dot = fmaf(q[2 * e], bf2f((bf16)(kw[t][e] & 0xFFFFu)), dot);
          dot = fmaf(q[2 * e + 1], bf2f((bf16)(kw[t][e] >> 16)), dot);
        }
        dot = group_sum<LPH>(dot);
        sc[t] = (t < tn) ? dot * g.scale_log2 : -INFINITY;
        bmax = fmaxf(bmax, sc[t]);
      }
      const float mn = fmaxf(mt, bmax);
      const float alpha = (mt == -INFINITY) ? 0.f : fast_exp2(mt - mn);
      lt *= alpha;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] *= alpha;
#pragma unroll
      for (int t = 0; t < PB; ++t) {
        const float p = (t < tn) ? fast_exp2(sc[t] - mn) : 0.f;
        lt += p;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[2 * e] = fmaf(p, bf2f((bf16)(vw[t][e] & 0xFFFFu)), acc[2 * e]);
          acc[2 * e + 1] = fmaf(p, bf2f((bf16)(vw[t][e] >> 16)), acc[2 * e + 1]);
        }
      }
      mt = mn;
    }
    if (act) {
      const float inv = 1.f / lt;
      u32x4 ow;
#pragma unroll
      for (int e = 0; e < 4; ++e) ow[e] = pack2bf(acc[2 * e] * inv, acc[2 * e + 1] * inv);
      *(u32x4*)(O + ((long)r * g.H + head) * HD + dl * 8) = ow;
    }
  }
}

}  // namespace alr
