// Row-wise kernels (gfx950): embedding gather, RMSNorm, row gathers, weight
// repacking and the output-head finalisation (log-sum-exp, greedy argmax,
// in-place log-softmax).
#pragma once

#include "device_common.hpp"

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

// resid[r, :] = given[r, :] where mask[r] != 0, else E[tok[r], :]  (fp32 stream)
template <typename T>
__global__ __launch_bounds__(256) void embed_kernel(float* __restrict__ resid,
                                                    const int* __restrict__ tok,
                                                    const T* __restrict__ E,
                                                    const T* __restrict__ given,
                                                    const uint8_t* __restrict__ mask, int d) {
  const long r = blockIdx.x;
  const bool use_given = mask != nullptr && mask[r] != 0;
  const T* src = use_given ? given + r * d : E + (long)tok[r] * d;
  float* dst = resid + r * d;
  for (int c = threadIdx.x; c < d; c += blockDim.x) dst[c] = Elt<T>::ld(src + c);
}

// out[r, :] = x[r, :] * g / sqrt(mean(x[r, :]^2) + eps)
template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* __restrict__ x,
                                                      const T* __restrict__ g,
                                                      T* __restrict__ out, int d, float eps) {
  __shared__ float red[4];
  const long r = blockIdx.x;
  const float* xr = x + r * d;
  float ss = 0.f;
  for (int c = threadIdx.x * 4; c < d; c += blockDim.x * 4) {
    const f32x4 v = *(const f32x4*)(xr + c);
    ss += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
  }
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  T* o = out + r * d;
  for (int c = threadIdx.x * 4; c < d; c += blockDim.x * 4) {
    const f32x4 v = *(const f32x4*)(xr + c);
#pragma unroll
    for (int e = 0; e < 4; ++e) Elt<T>::st(o + c + e, v[e] * inv * Elt<T>::ld(g + c + e));
  }
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

// Output head finalisation for the sorted row r of rollout slot s.
//   row data: logits (fp32) at lp + perm[r] * row_stride, V entries, written by
//   the output-head GEMM.  Computes max, argmax (ties -> lowest id) and
//   sum(exp(z - max)) in one pass, then overwrites the row with z - LSE.
//   tokens_out[perm[r] * block + s] = argmax; the next input token of row r is
//   forced[perm[r] * block + s] if that is >= 0, else the argmax.
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

__global__ __launch_bounds__(256) void lm_finalize_kernel(float* __restrict__ lp, long row_stride,
                                                          const int* __restrict__ perm, int V,
                                                          int* __restrict__ tokens_out, int block,
                                                          int s, const int* __restrict__ forced,
                                                          int* __restrict__ next_tok) {
  __shared__ MaxArg red[4];
  __shared__ float lse_sh;
  const int r = blockIdx.x;
  const long orow = perm[r];
  float* z = lp + orow * row_stride;
  MaxArg acc = {-INFINITY, 0.f, 0x7FFFFFFF};
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
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    MaxArg b;
    b.m = __shfl_xor(acc.m, o);
    b.s = __shfl_xor(acc.s, o);
    b.i = __shfl_xor(acc.i, o);
    acc = merge_maxarg(acc, b);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    MaxArg t = red[0];
    for (int w = 1; w < (int)(blockDim.x >> 6); ++w) t = merge_maxarg(t, red[w]);
    lse_sh = t.m + logf(t.s);
    tokens_out[orow * block + s] = t.i;
    int nxt = t.i;
    if (forced != nullptr) {
      const int f = forced[orow * block + s];
      if (f >= 0) nxt = f;
    }
    next_tok[r] = nxt;
  }
  __syncthreads();
  const float lse = lse_sh;
  for (int c = threadIdx.x * 4; c < V; c += blockDim.x * 4) {
    f32x4 v = *(const f32x4*)(z + c);
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] -= lse;
    *(f32x4*)(z + c) = v;
  }
}

}  // namespace alr
