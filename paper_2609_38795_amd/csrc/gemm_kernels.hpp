// GEMM kernels C[M,N] = A[M,K] * W[N,K]^T with fused epilogues (gfx950).
//
// bf16 path: 32x32x16 bf16 MFMA, 128x128x64 workgroup tile, 4 waves as 2x2,
// each wave a 64x64 sub-tile (2x2 MFMA blocks).  fp32 path: FMA, 64x64x16
// tile.  Both hand the epilogue *pairs* of outputs: the value at column c and
// the one at column c+32, where c lies in the low half of a 64-column group.
// Weight rows are arranged at context creation so that every fused operation
// needs exactly such a pair: SwiGLU's gate/up values and RoPE's rotate-half
// partners (i, i + head_dim/2) land 32 columns apart in the same lane.
#pragma once

#include "device_common.hpp"

namespace alr {

// ------------------------------------------------------------------ epilogues

// QKV projection + RoPE + key/value store.  Columns [0, H*hd) are q, then
// [H*hd, H*hd+G*hd) k, then v.  In the q and k sections, 64-column group t
// holds, in its low half, entries f = 32t .. 32t+31 of the list of
// first-half dimensions (head = f / (hd/2), i = f % (hd/2)) and, in its high
// half, their partners i + hd/2.  Outputs are written in natural order.
template <typename OutT>
struct EpiQKV {
  OutT* q;            // [M, H*hd]
  OutT* k;            // row r -> k + r*kv_rs
  OutT* v;            // row r -> v + r*kv_rs
  long kv_rs;
  const float* cosT;  // [max_pos, hd/2]
  const float* sinT;
  const int* pos;     // position of row r is pos[r] + pos_add
  int pos_add;
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
      const long p = (long)(pos[row] + pos_add);
      const float cs = cosT[p * half + i], sn = sinT[p * half + i];
      Elt<OutT>::st(dst + head * hd + i, lo * cs - hi * sn);
      Elt<OutT>::st(dst + head * hd + i + half, hi * cs + lo * sn);
    } else {
      OutT* dst = v + (long)row * kv_rs;
      const int cl = c - qd - kd;
      Elt<OutT>::st(dst + cl, lo);
      Elt<OutT>::st(dst + cl + 32, hi);
    }
  }
};

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
};

// SwiGLU: 64-column group t holds gate rows 32t..32t+31 then up rows
// 32t..32t+31; out[row, 32t + w] = SiLU(gate) * up.
template <typename OutT>
struct EpiSwiGLU {
  OutT* out;
  int ld;
  __device__ __forceinline__ void operator()(int row, int c, float g, float u) const {
    const int col = (c >> 6) * 32 + (c & 63);
    const float s = g / (1.0f + expf(-g));
    Elt<OutT>::st(out + (long)row * ld + col, s * u);
  }
};

// Plain fp32 store of logits into caller rows: out + (perm ? perm[row] : row) * rs.
struct EpiLogits {
  float* out;
  long rs;
  const int* perm;
  __device__ __forceinline__ void operator()(int row, int c, float lo, float hi) const {
    const long r = perm ? perm[row] : row;
    float* p = out + r * rs + c;
    p[0] = lo;
    p[32] = hi;
  }
};

// ------------------------------------------------------------------ bf16 MFMA GEMM

constexpr int GB_M = 128, GB_N = 128, GB_K = 64;
constexpr int GB_PITCH = GB_K + 8;  // bf16 elements per LDS row (144 bytes)

// Tile order: workgroups are dispatched round-robin over the 8 XCDs, so the
// block id is first remapped to make each XCD walk a contiguous range of the
// tile order; the order itself groups 8 M-tiles per N sweep so neighbouring
// tiles share A rows and W rows in L2.
__device__ __forceinline__ void gemm_tile_coords(int tiles_m, int tiles_n, int& tm, int& tn) {
  const int nb = tiles_m * tiles_n;
  int bid = blockIdx.x;
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

// TAG only separates the instantiations of different call sites, so that
// profilers report each GEMM of the model on its own line.
template <int TAG, class Epi>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(const bf16* __restrict__ A, int lda,
                                                        const bf16* __restrict__ W, int ldw,
                                                        int M, int N, int K, int tiles_m,
                                                        int tiles_n, Epi epi) {
  __shared__ __attribute__((aligned(16))) bf16 As[GB_M * GB_PITCH];
  __shared__ __attribute__((aligned(16))) bf16 Ws[GB_N * GB_PITCH];
  int tm, tn;
  gemm_tile_coords(tiles_m, tiles_n, tm, tn);
  const int m0 = tm * GB_M, n0 = tn * GB_N;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // global -> register staging: 4 chunks of 16 bytes per operand per thread
  u32x4 ra[4], rw[4];
  const bf16* a_src[4];
  const bf16* w_src[4];
  int lds_off[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ch = tid + 256 * i;
    const int r = ch >> 3, c8 = (ch & 7) * 8;
    const int ar = min(m0 + r, M - 1), wr = min(n0 + r, N - 1);
    a_src[i] = A + (long)ar * lda + c8;
    w_src[i] = W + (long)wr * ldw + c8;
    lds_off[i] = r * GB_PITCH + c8;
  }
  const int nk = K / GB_K;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ra[i] = *(const u32x4*)(a_src[i]);
    rw[i] = *(const u32x4*)(w_src[i]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    *(u32x4*)(As + lds_off[i]) = ra[i];
    *(u32x4*)(Ws + lds_off[i]) = rw[i];
  }
  __syncthreads();

  f32x16 acc[2][2];
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.f;

  const int lr = lane & 31, lk = (lane >> 5) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) {
      const int ko = (kt + 1) * GB_K;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ra[i] = *(const u32x4*)(a_src[i] + ko);
        rw[i] = *(const u32x4*)(w_src[i] + ko);
      }
    }
#pragma unroll
    for (int ks = 0; ks < GB_K / 16; ++ks) {
      bf16x8 av[2], bv[2];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
        av[mi] = as_bf16x8(*(const u32x4*)(As + (wm * 64 + mi * 32 + lr) * GB_PITCH + ks * 16 + lk));
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
        bv[ni] = as_bf16x8(*(const u32x4*)(Ws + (wn * 64 + ni * 32 + lr) * GB_PITCH + ks * 16 + lk));
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) acc[mi][ni] = mfma32x32x16(av[mi], bv[ni], acc[mi][ni]);
    }
    __syncthreads();
    if (kt + 1 < nk) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        *(u32x4*)(As + lds_off[i]) = ra[i];
        *(u32x4*)(Ws + lds_off[i]) = rw[i];
      }
    }
    __syncthreads();
  }

  const int col = n0 + wn * 64 + lr;
  if (col < N) {
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 64 + mi * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (row < M) epi(row, col, acc[mi][0][r], acc[mi][1][r]);
      }
  }
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
