// Row-wise kernels (gfx950): embedding gather, RMSNorm, row gathers, weight
// repacking and the output-head finalisation (log-sum-exp, greedy argmax,
// in-place log-softmax).
#pragma once

#include "device_common.hpp"
#include "gemm_kernels.hpp"

namespace alr {

__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float t = 0.f;
  const int nw = blockDim.x >> 6;
  for (int i = 0; i < nw; ++i) t += red[i];
  __syncthreads();
  return t;
}

// resid[r, :] = given[r, :] where mask[r] != 0, else E[tok[r], :]  (fp32 stream);
// d a multiple of 16 / sizeof(T).  Each thread moves 16-byte chunks of the
// source row, four at a time: the loads of a round are issued before its
// stores, so a row costs a round trip per 4 x 256 chunks, not per element.
template <typename T>
__global__ __launch_bounds__(256) void embed_kernel(float* __restrict__ resid,
                                                    const int* __restrict__ tok,
                                                    const T* __restrict__ E,
                                                    const T* __restrict__ given,
                                                    const uint8_t* __restrict__ mask, int d) {
  constexpr int EPC = 16 / (int)sizeof(T);  // elements per 16-byte chunk
  constexpr int U = 4;                      // chunks per thread per round
  const long r = blockIdx.x;
  const bool use_given = mask != nullptr && mask[r] != 0;
  const T* src = use_given ? given + r * d : E + (long)tok[r] * d;
  float* dst = resid + r * d;
  const int nch = d / EPC;
  for (int c0 = threadIdx.x; c0 < nch; c0 += 256 * U) {
    u32x4 w[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (c0 + 256 * u < nch) w[u] = *(const u32x4*)(src + (long)(c0 + 256 * u) * EPC);
    __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));  // vmcnt(0): the round's loads landed
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + 256 * u;
      if (c >= nch) continue;
      float* o = dst + (long)c * EPC;
      if constexpr (sizeof(T) == 4) {
        *(u32x4*)o = w[u];
      } else {
        f32x4 a, b;
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          a[2 * e] = __uint_as_float(w[u][e] << 16);
          a[2 * e + 1] = __uint_as_float(w[u][e] & 0xFFFF0000u);
          b[2 * e] = __uint_as_float(w[u][2 + e] << 16);
          b[2 * e + 1] = __uint_as_float(w[u][2 + e] & 0xFFFF0000u);
        }
        *(f32x4*)o = a;
        *(f32x4*)(o + 4) = b;
      }
    }
  }
}

// Four gain elements held in registers (fp32, or bf16 bit patterns)
template <typename T>
struct Gain4;
template <>
struct Gain4<float> {
  f32x4 v;
  __device__ __forceinline__ void load(const float* g) { v = *(const f32x4*)g; }
  __device__ __forceinline__ float operator[](int e) const { return v[e]; }
};
template <>
struct Gain4<bf16> {
  u32x2 w;
  __device__ __forceinline__ void load(const bf16* g) { w = *(const u32x2*)g; }
  __device__ __forceinline__ float operator[](int e) const {
    return bf2f((bf16)((e & 1) ? w[e >> 1] >> 16 : w[e >> 1] & 0xFFFFu));
  }
};

// out[c .. c+3] = v * inv * g[c .. c+3], four elements at once
__device__ __forceinline__ void norm4(float* o, f32x4 v, const Gain4<float>& g, float inv) {
  f32x4 w;
#pragma unroll
  for (int e = 0; e < 4; ++e) w[e] = v[e] * inv * g[e];
  *(f32x4*)o = w;
}
__device__ __forceinline__ void norm4(bf16* o, f32x4 v, const Gain4<bf16>& g, float inv) {
  u32x2 w;
  w[0] = pack2bf(v[0] * inv * g[0], v[1] * inv * g[1]);
  w[1] = pack2bf(v[2] * inv * g[2], v[3] * inv * g[3]);
  *(u32x2*)o = w;
}

// out[r, :] = x[r, :] * g / sqrt(mean(x[r, :]^2) + eps); d a multiple of 4.  The
// row and its gains stay in registers between the two passes for d <= 8192.
// Every load of the row and of the gains is issued before the first use, so a
// row costs one memory round trip instead of one per chunk (a load followed by
// its use in the same conditional block makes the compiler wait there).
template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* __restrict__ x,
                                                      const T* __restrict__ g,
                                                      T* __restrict__ out, int d, float eps) {
  constexpr int CACHE = 8;  // 4-element chunks per thread held in registers
  __shared__ float red[4];
  const long r = blockIdx.x;
  const float* xr = x + r * d;
  T* o = out + r * d;
  f32x4 v[CACHE];
  Gain4<T> gv[CACHE];
#pragma unroll
  for (int k = 0; k < CACHE; ++k) {
    const int c = (threadIdx.x + 256 * k) * 4;
    if (c < d) {
      v[k] = *(const f32x4*)(xr + c);
      gv[k].load(g + c);
    }
  }
  // vmcnt(0): the loads of every chunk have landed.  Without it the compiler
  // cannot tell at the conditional stores below whether a gain load is still
  // outstanding and waits before each store, and on this target such a wait
  // also waits for the previous store.
  __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < CACHE; ++k) {
    const int c = (threadIdx.x + 256 * k) * 4;
    if (c < d) ss += v[k][0] * v[k][0] + v[k][1] * v[k][1] + v[k][2] * v[k][2] + v[k][3] * v[k][3];
  }
  for (int c = (threadIdx.x + 256 * CACHE) * 4; c < d; c += 1024) {
    const f32x4 w = *(const f32x4*)(xr + c);
    ss += w[0] * w[0] + w[1] * w[1] + w[2] * w[2] + w[3] * w[3];
  }
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
  for (int k = 0; k < CACHE; ++k) {
    const int c = (threadIdx.x + 256 * k) * 4;
    if (c < d) norm4(o + c, v[k], gv[k], inv);
  }
  for (int c = (threadIdx.x + 256 * CACHE) * 4; c < d; c += 1024) {
    Gain4<T> gt;
    gt.load(g + c);
    norm4(o + c, *(const f32x4*)(xr + c), gt, inv);
  }
}

// The reduce of a split-K residual update fused with the RMSNorm that reads the
// updated residual, one workgroup per row of d <= 1024 CH elements:
//   h[r, :] += part[0, r, :] + ... + part[S-1, r, :]
// (the slices added in slice order and the sum then added to h, as
// splitk_reduce_kernel with EpiResid does), the updated row copied to feature
// row perm[r] (or r) when feat is set, and out[r, :] = RMSNorm(h[r, :]) * g with
// the element order, sums and rounding of rmsnorm_kernel.  Every load of the
// row (partials, residual, gains) is issued before the first add.
template <typename T, int S, int CH>
__global__ __launch_bounds__(256) void splitk_resid_norm_kernel(
    const float* __restrict__ part, long sstride, float* __restrict__ h, float* __restrict__ feat,
    long feat_rs, const int* __restrict__ perm, const T* __restrict__ g, T* __restrict__ out,
    int d, float eps) {
  __shared__ float red[4];
  const long r = blockIdx.x;
  float* hr = h + r * d;
  const float* pr = part + r * d;
  f32x4 v[CH], ps[CH][S];
  Gain4<T> gv[CH];
#pragma unroll
  for (int k = 0; k < CH; ++k) {
    const int c = (threadIdx.x + 256 * k) * 4;
    if (c < d) {
      v[k] = *(const f32x4*)(hr + c);
#pragma unroll
      for (int sl = 0; sl < S; ++sl) ps[k][sl] = *(const f32x4*)(pr + sl * sstride + c);
      gv[k].load(g + c);
    }
  }
  __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));  // vmcnt(0), as in rmsnorm_kernel
  float* fr = feat ? feat + (perm ? (long)perm[r] : r) * feat_rs : nullptr;
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < CH; ++k) {
    const int c = (threadIdx.x + 256 * k) * 4;
    if (c < d) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float acc = 0.f;
#pragma unroll
        for (int sl = 0; sl < S; ++sl) acc += ps[k][sl][e];
        v[k][e] = v[k][e] + acc;
      }
      *(f32x4*)(hr + c) = v[k];
      if (fr) *(f32x4*)(fr + c) = v[k];
      ss += v[k][0] * v[k][0] + v[k][1] * v[k][1] + v[k][2] * v[k][2] + v[k][3] * v[k][3];
    }
  }
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
  for (int k = 0; k < CH; ++k) {
    const int c = (threadIdx.x + 256 * k) * 4;
    if (c < d) norm4(out + r * d + c, v[k], gv[k], inv);
  }
}

// Row-major assembly from a table of source rows: dst row n = src[n] (K bf16
// elements, K a multiple of 8); used to build the fused weight matrices.
__global__ __launch_bounds__(256) void gather_rows_ptr_kernel(bf16* __restrict__ dst,
                                                              const bf16* const* __restrict__ src,
                                                              int N, int K) {
  const long q = (long)blockIdx.x * 256 + threadIdx.x;  // 16-byte chunk index
  const int cpr = K / 8;
  if (q >= (long)N * cpr) return;
  const int n = (int)(q / cpr), c = (int)(q % cpr);
  *(u32x4*)(dst + q * 8) = *(const u32x4*)(src[n] + c * 8);
}

// dst[r, :] = src[idx[r], :]  (row_elems elements of T)
template <typename T>
__global__ __launch_bounds__(256) void gather_rows_kernel(T* __restrict__ dst,
                                                          const T* __restrict__ src,
                                                          const int* __restrict__ idx,
                                                          long row_elems) {
  const long r = blockIdx.x;
  const T* s = src + (long)idx[r] * row_elems;
  T* o = dst + r * row_elems;
  for (long c = threadIdx.x; c < row_elems; c += blockDim.x) o[c] = s[c];
}

// Slot-0 features: dst[perm[r]] (row stride dst_rs) = src[idx[r]] (n elements)
__global__ __launch_bounds__(256) void gather_feat_kernel(float* __restrict__ dst, long dst_rs,
                                                          const int* __restrict__ perm,
                                                          const float* __restrict__ src,
                                                          const int* __restrict__ idx, long n) {
  const long r = blockIdx.x;
  const float* s = src + (long)idx[r] * n;
  float* o = dst + (long)perm[r] * dst_rs;
  for (long c = threadIdx.x * 4; c < n; c += blockDim.x * 4) *(f32x4*)(o + c) = *(const f32x4*)(s + c);
}

// Weight repacking: dst row dst_row[r] = src row r (row_bytes, multiple of 16).
__global__ __launch_bounds__(256) void scatter_rows_kernel(char* __restrict__ dst,
                                                           const char* __restrict__ src,
                                                           const int* __restrict__ dst_row,
                                                           long row_bytes) {
  const long r = blockIdx.x;
  const u32x4* s = (const u32x4*)(src + r * row_bytes);
  u32x4* o = (u32x4*)(dst + (long)dst_row[r] * row_bytes);
  for (long c = threadIdx.x; c < row_bytes / 16; c += blockDim.x) o[c] = s[c];
}

// Output head finalisation of the sorted row r of slot s.
//   Logits (fp32, V entries) of row r are at z + (z_perm ? perm[r] : r) * z_rs,
//   written by the output-head GEMM.  Outputs go to index o = perm[r] * block + s
//   (the caller's anchor order).  The row's max and sum(exp(z - max)) come from
//   the GEMM epilogue's per-group partials (part[r * part_ld + g], g < part_ld =
//   V / 64) when part is set, and the argmax (ties -> lowest id) is then the
//   first column equal to the max, found in the pass below; without partials a
//   first pass over the logits gives all three.  Then one pass rewrites the row
//   as z - LSE (write_lp) and, with TOPK, keeps each thread's 8 best (value, id)
//   pairs, ranked by decreasing value and then increasing id, while summing
//   exp(z - max) over every entry the thread drops from (or never admits to)
//   that list; eight block-wide argmax rounds merge the lists into the row's
//   top 8, and the entries left in the lists join the sum, which is then the
//   mass of exactly the tokens ranked after the 8th (the tail bucket).
//   next_tok[r] = forced[o] if that is >= 0, else the argmax.  target_logp[o]
//   = log p(target[r]) (nan when target[r] < 0).  A row with valid[r] == 0 gets
//   token -1, top ids -1, top log-probs -inf, tail 0, target log-prob nan and,
//   when write_lp, a row of -inf.
constexpr int ALR_K_TOP = 8;

struct LmFinalize {
  float* z;
  long z_rs;
  int z_perm;
  int write_lp;
  const int* perm;
  int V, block, s;
  int* tokens;         // [o] or null
  const int* forced;   // [o] or null
  int* next_tok;       // [r] or null
  int* top_ids;        // [o * 8] (TOPK)
  float* top_logp;     // [o * 8] (TOPK)
  float* tail;         // [o] (TOPK)
  const int* target;   // [r] or null
  float* target_logp;  // [o] (with target)
  const unsigned char* valid;  // [r] or null
  const LogitPart* part;       // [r * part_ld + g] or null
  int part_ld;
};

struct MaxArg {
  float m, s;
  int i;
};
__device__ __forceinline__ MaxArg merge_maxarg(MaxArg a, MaxArg b) {
  if (b.m > a.m || (b.m == a.m && b.i < a.i)) {
    const float sa = (a.m == -INFINITY) ? 0.f : a.s * expf(a.m - b.m);
    return {b.m, sa + b.s, b.i};
  }
  const float sb = (b.m == -INFINITY) ? 0.f : b.s * expf(b.m - a.m);
  return {a.m, a.s + sb, a.i};
}

// (v, i) ranks before (w, j): larger value, then lower id
__device__ __forceinline__ bool ranks_before(float v, int i, float w, int j) {
  return v > w || (v == w && i < j);
}

template <bool TOPK>
__global__ __launch_bounds__(256) void lm_finalize_kernel(LmFinalize a) {
  __shared__ MaxArg red[4];
  __shared__ float lse_sh, m_sh, s_sh, tgt_sh;
  __shared__ float win_v[4], top_v[ALR_K_TOP];
  __shared__ int win_i[4], top_i[ALR_K_TOP];
  __shared__ float tail_red[4];
  const int r = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const long orow = a.perm[r];
  const long o = orow * a.block + a.s;
  float* z = a.z + (a.z_perm ? orow : (long)r) * a.z_rs;
  const int V = a.V;
  if (a.valid != nullptr && a.valid[r] == 0) {  // uniform over the block
    if (threadIdx.x == 0) {
      if (a.tokens) a.tokens[o] = -1;
      if (a.next_tok) a.next_tok[r] = 0;
      if (a.target) a.target_logp[o] = __builtin_nanf("");
      if (TOPK) a.tail[o] = 0.f;
    }
    if (TOPK && threadIdx.x < ALR_K_TOP) {
      a.top_ids[o * ALR_K_TOP + threadIdx.x] = -1;
      a.top_logp[o * ALR_K_TOP + threadIdx.x] = -INFINITY;
    }
    if (a.write_lp)
      for (int c = threadIdx.x; c < V; c += blockDim.x) z[c] = -INFINITY;
    return;
  }
  MaxArg acc = {-INFINITY, 0.f, 0x7FFFFFFF};
  const bool from_part = a.part != nullptr;
  // Loads go out four at a time before their uses (one memory round trip per
  // four, where a load used in the same iteration costs one each); every
  // thread still visits its groups and columns in increasing order.
  constexpr int U = 4;
  if (from_part) {
    const LogitPart* pr = a.part + (long)r * a.part_ld;
    for (int g0 = threadIdx.x; g0 < a.part_ld; g0 += blockDim.x * U) {
      LogitPart q[U];
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (g0 + u * (int)blockDim.x < a.part_ld) q[u] = pr[g0 + u * blockDim.x];
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (g0 + u * (int)blockDim.x < a.part_ld)
          acc = merge_maxarg(acc, MaxArg{q[u].m, q[u].s, 0x7FFFFFFF});
    }
  } else {
    for (int c = threadIdx.x * 4; c < V; c += blockDim.x * 4) {
      const f32x4 v = *(const f32x4*)(z + c);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (v[e] > acc.m) {
          acc.s = (acc.m == -INFINITY) ? 1.f : acc.s * expf(acc.m - v[e]) + 1.f;
          acc.m = v[e];
          acc.i = c + e;
        } else {
          acc.s += expf(v[e] - acc.m);
        }
      }
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    MaxArg b;
    b.m = __shfl_xor(acc.m, off);
    b.s = __shfl_xor(acc.s, off);
    b.i = __shfl_xor(acc.i, off);
    acc = merge_maxarg(acc, b);
  }
  if (lane == 0) red[wave] = acc;
  __syncthreads();
  // the greedy token (or the forced one) goes out once the argmax is known
  auto emit_token = [&](int arg) {
    if (a.tokens) a.tokens[o] = arg;
    if (a.next_tok) {
      int nxt = arg;
      if (a.forced != nullptr) {
        const int f = a.forced[o];
        if (f >= 0) nxt = f;
      }
      a.next_tok[r] = nxt;
    }
  };
  if (threadIdx.x == 0) {
    MaxArg t = red[0];
    for (int w = 1; w < (int)(blockDim.x >> 6); ++w) t = merge_maxarg(t, red[w]);
    lse_sh = t.m + logf(t.s);
    m_sh = t.m;
    s_sh = t.s;
    if (!from_part) emit_token(t.i);
    if (a.target) {
      const int x = a.target[r];
      tgt_sh = (x >= 0) ? z[x] : __builtin_nanf("");
    }
  }
  __syncthreads();
  const float lse = lse_sh, m = m_sh;
  if (!a.write_lp && !TOPK && !from_part) {
    if (a.target && threadIdx.x == 0) a.target_logp[o] = tgt_sh - lse;
    return;
  }
  float tv[ALR_K_TOP];
  int ti[ALR_K_TOP];
#pragma unroll
  for (int j = 0; j < ALR_K_TOP; ++j) {
    tv[j] = -INFINITY;
    ti[j] = 0x7FFFFFFF;
  }
  float tsum = 0.f;  // exp(z - m) of the entries this thread dropped or never admitted
  int arg = 0x7FFFFFFF;  // this thread's first column equal to the row max
  const int cstep = blockDim.x * 4;
  if constexpr (!TOPK) {
    // no data-dependent branch in the source: the loads of a round are
    // unconditional (a column past V re-reads the row's last chunk, unused)
    // and the argmax update is a select
    for (int c0 = threadIdx.x * 4; c0 < V; c0 += cstep * U) {
      f32x4 vv[U];
#pragma unroll
      for (int u = 0; u < U; ++u) vv[u] = *(const f32x4*)(z + min(c0 + u * cstep, V - 4));
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c = c0 + u * cstep;
        const bool in = c < V;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          arg = (in && arg == 0x7FFFFFFF && vv[u][e] == m) ? c + e : arg;  // columns rise
          vv[u][e] -= lse;
        }
        if (in && a.write_lp) *(f32x4*)(z + c) = vv[u];
      }
    }
  } else {
    for (int c0 = threadIdx.x * 4; c0 < V; c0 += cstep * U) {
      f32x4 vv[U];
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (c0 + u * cstep < V) vv[u] = *(const f32x4*)(z + c0 + u * cstep);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c = c0 + u * cstep;
        if (c >= V) break;
        f32x4 v = vv[u];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (arg == 0x7FFFFFFF && v[e] == m) arg = c + e;  // columns rise within a thread
          // this thread meets ids in increasing order, so an equal value ranks
          // after the entries already held: admit only strictly larger values
          if (v[e] > tv[ALR_K_TOP - 1]) {
            const float out_v = tv[ALR_K_TOP - 1];
            if (out_v != -INFINITY) tsum += expf(out_v - m);
            float pv = v[e];
            int pi = c + e;
            bool sh = false;
#pragma unroll
            for (int j = 0; j < ALR_K_TOP; ++j) {
              const bool take = sh || (v[e] > tv[j]);
              if (take) {
                const float ov = tv[j];
                const int oi = ti[j];
                tv[j] = pv;
                ti[j] = pi;
                pv = ov;
                pi = oi;
              }
              sh = take;
            }
          } else {
            tsum += expf(v[e] - m);
          }
          v[e] -= lse;
        }
        if (a.write_lp) *(f32x4*)(z + c) = v;
      }
    }
  }
  if (from_part) {  // lowest column holding the max over the block
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) arg = min(arg, __shfl_xor(arg, off));
    if (lane == 0) win_i[wave] = arg;
    __syncthreads();
    if (threadIdx.x == 0) {
      int t = win_i[0];
      for (int w = 1; w < (int)(blockDim.x >> 6); ++w) t = min(t, win_i[w]);
      emit_token(t);
    }
    __syncthreads();  // win_i is reused by the top-8 rounds
  }
  if constexpr (TOPK) {
    // eight rounds: the best head of all threads' lists is the next entry
    for (int k = 0; k < ALR_K_TOP; ++k) {
      float bv = tv[0];
      int bi = ti[0];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const float ov = __shfl_xor(bv, off);
        const int oi = __shfl_xor(bi, off);
        if (ranks_before(ov, oi, bv, bi)) {
          bv = ov;
          bi = oi;
        }
      }
      if (lane == 0) {
        win_v[wave] = bv;
        win_i[wave] = bi;
      }
      __syncthreads();
      if (threadIdx.x == 0) {
        float wv = win_v[0];
        int wi = win_i[0];
        for (int w = 1; w < (int)(blockDim.x >> 6); ++w)
          if (ranks_before(win_v[w], win_i[w], wv, wi)) {
            wv = win_v[w];
            wi = win_i[w];
          }
        top_v[k] = wv;
        top_i[k] = wi;
      }
      __syncthreads();
      if (ti[0] == top_i[k] && tv[0] != -INFINITY) {  // ids are unique: the owner pops its head
#pragma unroll
        for (int j = 0; j < ALR_K_TOP - 1; ++j) {
          tv[j] = tv[j + 1];
          ti[j] = ti[j + 1];
        }
        tv[ALR_K_TOP - 1] = -INFINITY;
        ti[ALR_K_TOP - 1] = 0x7FFFFFFF;
      }
    }
    // what is left in the lists ranks after the 8th entry
#pragma unroll
    for (int j = 0; j < ALR_K_TOP; ++j)
      if (tv[j] != -INFINITY) tsum += expf(tv[j] - m);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) tsum += __shfl_xor(tsum, off);
    if (lane == 0) tail_red[wave] = tsum;
    __syncthreads();
    if (threadIdx.x == 0) {
      float t = 0.f;
      for (int w = 0; w < (int)(blockDim.x >> 6); ++w) t += tail_red[w];
      a.tail[o] = t / s_sh;
    }
    if (threadIdx.x < ALR_K_TOP) {
      const bool have = top_v[threadIdx.x] != -INFINITY;
      a.top_ids[o * ALR_K_TOP + threadIdx.x] = have ? top_i[threadIdx.x] : -1;
      a.top_logp[o * ALR_K_TOP + threadIdx.x] = have ? top_v[threadIdx.x] - lse : -INFINITY;
    }
  }
  if (a.target && threadIdx.x == 0) a.target_logp[o] = tgt_sh - lse;
}

// Zero the entries of the transposed V cache that pad each sequence to a
// multiple of 64 keys: attention tiles copy them into LDS, and their
// probabilities being 0 keeps them out of the sums only if they hold finite
// values.  pad[2 s] is sequence s's first padding key column, pad[2 s + 1] the
// number of padding keys (< 64); key column k is stored at vt_perm(k).  Thread
// t covers sequence t % n_seq, cache row (t / n_seq) % rows, layer t / (n_seq rows).
__global__ __launch_bounds__(256) void zero_vt_pad_kernel(bf16* __restrict__ vc,
                                                          long layer_elems, long vt_stride,
                                                          const int* __restrict__ pad, int n_seq,
                                                          int rows, long total) {
  const long t = (long)blockIdx.x * 256 + threadIdx.x;
  if (t >= total) return;
  const int sq = (int)(t % n_seq);
  const long rl = t / n_seq;
  const int row = (int)(rl % rows);
  const long layer = rl / rows;
  bf16* p = vc + layer * layer_elems + (long)row * vt_stride;
  for (int c = 0; c < pad[2 * sq + 1]; ++c) p[vt_perm(pad[2 * sq] + c)] = 0;
}

// Corpus-label rows of slot s: row r takes the prefill's final-norm row at
// position min(a + s, len - 1) of its sequence (a = apos[r], len = alen[r],
// first token row atok[r] - apos[r]); valid[r] = (a + s <= len - 1);
// target[r] = the corpus token at a + s + 1 (from ctok, -1 for a given input
// row) when a + s + 1 <= len - 1, else -1.
template <typename T>
__global__ __launch_bounds__(256) void corpus_rows_kernel(T* __restrict__ dst,
                                                          const T* __restrict__ src,
                                                          const int* __restrict__ atok,
                                                          const int* __restrict__ apos,
                                                          const int* __restrict__ alen,
                                                          const int* __restrict__ ctok, int s,
                                                          long row_elems,
                                                          unsigned char* __restrict__ valid,
                                                          int* __restrict__ target) {
  const long r = blockIdx.x;
  const int a = apos[r], len = alen[r], t0 = atok[r] - a;
  const int p = min(a + s, len - 1);
  const T* sp = src + (long)(t0 + p) * row_elems;
  T* op = dst + r * row_elems;
  for (long c = threadIdx.x; c < row_elems; c += blockDim.x) op[c] = sp[c];
  if (threadIdx.x == 0) {
    valid[r] = (a + s <= len - 1) ? 1 : 0;
    target[r] = (a + s + 1 <= len - 1) ? ctok[t0 + a + s + 1] : -1;
  }
}

// Erase gates of anchor row r (caller order o = perm[r]) from the per-slot
// corpus log-probs and argmax tokens written by lm_finalize_kernel:
// soft[s] = exp(sum_{t<s} lp[t]), hard[s] = prod_{t<s} [argmax[t] == x_{a+t+1}];
// a slot past the sequence end gets 0 and so does everything after a factor
// that is undefined (nan log-prob).
__global__ __launch_bounds__(256) void erase_gates_kernel(const int* __restrict__ perm,
                                                          const int* __restrict__ atok,
                                                          const int* __restrict__ apos,
                                                          const int* __restrict__ alen,
                                                          const int* __restrict__ ctok,
                                                          const float* __restrict__ clp,
                                                          const int* __restrict__ amax, int n,
                                                          int block, float* __restrict__ soft,
                                                          float* __restrict__ hard) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= n) return;
  const long o0 = (long)perm[r] * block;
  const int a = apos[r], len = alen[r], t0 = atok[r] - a;
  float cum = 0.f, h = 1.f;
  bool alive = true;
  for (int s = 0; s < block; ++s) {
    if (a + s > len - 1) {
      soft[o0 + s] = 0.f;
      hard[o0 + s] = 0.f;
      continue;
    }
    soft[o0 + s] = alive ? expf(cum) : 0.f;
    hard[o0 + s] = alive ? h : 0.f;
    const float lp = clp[o0 + s];
    if (!(lp == lp)) {  // nan: no corpus token follows
      alive = false;
    } else {
      cum += lp;
      h = (amax[o0 + s] == ctok[t0 + a + s + 1]) ? h : 0.f;
    }
  }
}

// Secondary blocks of in-rollout anchors: secondary q sits at offset j = off[q]
// of primary block p = prim[q] (1 <= j <= block-1).  token0[q] = tokens[p, j-1]
// (y*_j); its index s' copies the primary's labels at index j + s' while that
// is <= block-1 (else ids -1, log-probs -inf, tail 0); weight[q, s'] =
// exp(-s'/gamma) when j + s' + 1 <= block - 1 and (eos_id >= 0) the primary
// fed no EOS before index j + s', else 0.  One thread per (q, s').
__global__ __launch_bounds__(256) void ira_assemble_kernel(
    const int* __restrict__ prim, const int* __restrict__ off, int n_sec, int block,
    const int* __restrict__ tokens, const int* __restrict__ top_ids,
    const float* __restrict__ top_logp, const float* __restrict__ tail, float gamma, int eos_id,
    int* __restrict__ token0, int* __restrict__ s_ids, float* __restrict__ s_logp,
    float* __restrict__ s_tail, float* __restrict__ s_weight) {
  const long t = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (long)n_sec * block) return;
  const int q = (int)(t / block), s2 = (int)(t % block);
  const int p = prim[q], j = off[q];
  if (s2 == 0) token0[q] = tokens[(long)p * block + j - 1];
  const long dst = (long)q * block + s2;
  const int src = j + s2;
  if (src <= block - 1) {
    const long so = (long)p * block + src;
    for (int e = 0; e < ALR_K_TOP; ++e) {
      s_ids[dst * ALR_K_TOP + e] = top_ids[so * ALR_K_TOP + e];
      s_logp[dst * ALR_K_TOP + e] = top_logp[so * ALR_K_TOP + e];
    }
    s_tail[dst] = tail[so];
  } else {
    for (int e = 0; e < ALR_K_TOP; ++e) {
      s_ids[dst * ALR_K_TOP + e] = -1;
      s_logp[dst * ALR_K_TOP + e] = -INFINITY;
    }
    s_tail[dst] = 0.f;
  }
  bool alive = src <= block - 1;
  if (eos_id >= 0)  // the primary's slot src is masked once an EOS was fed before it
    for (int t = 0; t < src && t < block && alive; ++t)
      alive = tokens[(long)p * block + t] != eos_id;
  s_weight[dst] = (j + s2 + 1 <= block - 1 && alive) ? expf(-(float)s2 / gamma) : 0.f;
}

// Slot weights: w[i, s] = exp(-s / gamma) while no EOS occurs in tokens[i, 0 .. s-1],
// else 0.  One thread per block row.
__global__ __launch_bounds__(256) void slot_weights_kernel(const int* __restrict__ tokens,
                                                           int n, int block, int eos_id,
                                                           float gamma, float* __restrict__ w) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  bool alive = true;
  for (int s = 0; s < block; ++s) {
    w[(long)i * block + s] = alive ? expf(-(float)s / gamma) : 0.f;
    if (eos_id >= 0 && tokens[(long)i * block + s] == eos_id) alive = false;
  }
}

// Corpus tokens kept for the corpus labels: ctok[i] = tokens[i], or -1 where
// a given input row replaces the token (mask[i] != 0).
__global__ __launch_bounds__(256) void keep_tokens_kernel(int* __restrict__ ctok,
                                                          const int* __restrict__ tokens,
                                                          const unsigned char* __restrict__ mask,
                                                          int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) ctok[i] = (mask != nullptr && mask[i]) ? -1 : tokens[i];
}

}  // namespace alr
