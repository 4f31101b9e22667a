// Host runtime and C ABI of the anchor-branched greedy-rollout library.
//
// Call sequence per prefill (all sequences of the batch at once, M = total
// tokens): embed -> per layer [RMSNorm -> QKV GEMM (+RoPE, shared K/V store)
// -> causal attention -> O GEMM (+residual) -> RMSNorm -> gate|up GEMM
// (+SwiGLU) -> down GEMM (+residual, feature capture)] -> final RMSNorm.
//
// Call sequence per rollout: anchors are sorted by (sequence, position) so the
// decode attention can stream each sequence's shared keys once per group of
// anchors; slot 0 reads the prefill's final-norm row and features at the
// anchor; each later slot runs all anchors through the decoder as one batch
// (M = number of anchors), appending its key/value to the anchor's private
// buffer, and ends with the output-head GEMM and its finalisation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <functional>
#include <mutex>
#include <numeric>
#include <queue>
#include <string>
#include <type_traits>
#include <vector>

#include "../../include/alr.h"
#include "../../include/alr_debug.h"
#include "attn_kernels.hpp"
#include "gemm_kernels.hpp"
#include "misc_kernels.hpp"

using namespace alr;

static_assert(ALR_K_TOP == ALR_TOPK, "top-k size of the kernels and the ABI differ");

namespace {

thread_local std::string g_create_err;

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct Layout {
  size_t es;  // element size of the weight / operand dtype
  size_t w_embed, w_lm, w_fnorm;
  size_t layer0, layer_stride;  // per layer block
  size_t l_anorm, l_fnorm, l_qkv, l_o, l_gu, l_down;  // offsets within a layer block
  size_t rope_cos, rope_sin;
  size_t kc, vc, kv_layer_stride;
  size_t vt_stride;  // columns of the transposed V cache (0 when V is stored natural)
  size_t kp, vp, kvp_layer_stride;
  size_t feat_store, hf_store;
  size_t resid, xnorm, qbuf, attn, act;
  size_t i_tokpos, i_rowstart, i_perm, i_apos, i_rpos, i_atok, i_aseq, i_alen, i_cur;
  size_t i_valid, i_target, i_ira, i_ctok, logits, lm_part;
  size_t i_pwork, i_dwork, i_maps, i_vtcol, i_vtpad, i_rowinfo, i_rowptr;
  size_t part_o, part_ml;
  size_t splitk, splitk_bytes;
  size_t max_pwork, max_dwork, max_groups;
  size_t total;
};

bool fmt_msg(char* msg, size_t len, const char* f, ...) {
  if (msg && len) {
    va_list ap;
    va_start(ap, f);
    vsnprintf(msg, len, f, ap);
    va_end(ap);
  }
  return false;
}

alr_status check_config_impl(const alr_config* c, char* msg, size_t len) {
  if (!c) return fmt_msg(msg, len, "config is NULL"), ALR_E_INVALID_ARG;
  if (c->dtype != ALR_F32 && c->dtype != ALR_BF16)
    return fmt_msg(msg, len, "dtype %d is not ALR_F32 or ALR_BF16", c->dtype), ALR_E_INVALID_ARG;
  if (c->n_layers < 0 || c->d_model <= 0 || c->n_heads <= 0 || c->n_kv_heads <= 0 ||
      c->head_dim <= 0 || c->d_ffn <= 0 || c->vocab <= 0 || c->max_pos <= 0)
    return fmt_msg(msg, len, "non-positive dimension in config"), ALR_E_INVALID_ARG;
  if (!(c->rms_eps >= 0.f) || !(c->rope_base > 0.f))
    return fmt_msg(msg, len, "rms_eps must be >= 0 and rope_base > 0"), ALR_E_INVALID_ARG;
  if (c->n_heads % c->n_kv_heads != 0)
    return fmt_msg(msg, len, "n_heads %d is not a multiple of n_kv_heads %d", c->n_heads,
                   c->n_kv_heads),
           ALR_E_INVALID_ARG;
  const long q = (long)c->n_heads * c->head_dim, kv = (long)c->n_kv_heads * c->head_dim;
  if (c->d_model % 64 || c->d_ffn % 64 || q % 64 || kv % 64 || c->vocab % 64)
    return fmt_msg(msg, len,
                   "d_model, d_ffn, vocab, n_heads*head_dim and n_kv_heads*head_dim must be "
                   "multiples of 64"),
           ALR_E_UNSUPPORTED;
  if (c->head_dim % 2 || c->head_dim > 256 || (q / 2) % 32 || (kv / 2) % 32)
    return fmt_msg(msg, len,
                   "head_dim must be even and <= 256, and heads*head_dim/2 a multiple of 32"),
           ALR_E_UNSUPPORTED;
  {
    const int* ms = c->mrope_sections;
    const bool none = ms[0] == 0 && ms[1] == 0 && ms[2] == 0;
    if (!none && (ms[0] < 0 || ms[1] < 0 || ms[2] < 0 || ms[0] + ms[1] + ms[2] != c->head_dim / 2))
      return fmt_msg(msg, len, "mrope_sections (%d, %d, %d) must be all zero or non-negative with "
                               "sum head_dim/2 = %d", ms[0], ms[1], ms[2], c->head_dim / 2),
             ALR_E_INVALID_ARG;
  }
  if (c->n_feat < 0 || c->n_feat > ALR_MAX_FEAT)
    return fmt_msg(msg, len, "n_feat %d outside [0, %d]", c->n_feat, ALR_MAX_FEAT),
           ALR_E_INVALID_ARG;
  for (int i = 0; i < c->n_feat; ++i) {
    if (c->feat_layers[i] < 0 || c->feat_layers[i] >= c->n_layers)
      return fmt_msg(msg, len, "feat_layers[%d] = %d outside [0, n_layers)", i, c->feat_layers[i]),
             ALR_E_OUT_OF_RANGE;
    for (int j = 0; j < i; ++j)
      if (c->feat_layers[j] == c->feat_layers[i])
        return fmt_msg(msg, len, "feat_layers has duplicate layer %d", c->feat_layers[i]),
               ALR_E_INVALID_ARG;
  }
  return ALR_OK;
}

alr_status check_limits(const alr_limits* l, char* msg, size_t len) {
  if (!l) return fmt_msg(msg, len, "limits is NULL"), ALR_E_INVALID_ARG;
  if (l->max_tokens <= 0 || l->max_seqs <= 0 || l->max_anchors <= 0 || l->max_block <= 0)
    return fmt_msg(msg, len, "limits must be positive"), ALR_E_INVALID_ARG;
  return ALR_OK;
}

// The bf16 GEMM kernels address a thread's operand chunks by 32-bit byte
// offsets from the operand base, so every GEMM operand (activation rows of
// max(max_tokens, max_anchors) x K, weight matrices N x K) must stay below
// 4 GiB.  cfg and lim are already valid.
alr_status check_operand_sizes(const alr_config& c, const alr_limits& lim, char* msg, size_t len) {
  if (c.dtype != ALR_BF16) return ALR_OK;
  const double lim32 = 4294967296.0;
  const double d = c.d_model, F = c.d_ffn, V = c.vocab;
  const double qd = (double)c.n_heads * c.head_dim, kvd = (double)c.n_kv_heads * c.head_dim;
  const double R = std::max(lim.max_tokens, lim.max_anchors);
  const double act = R * std::max(std::max(d, F), qd) * 2.0;
  const double wmax = std::max(std::max(V * d, 2.0 * F * d), std::max((qd + 2 * kvd) * d, d * F)) * 2.0;
  if (act >= lim32)
    return fmt_msg(msg, len,
                   "GEMM activation operand of %.0f rows x %.0f bf16 is >= 4 GiB (lower max_tokens "
                   "/ max_anchors)",
                   R, std::max(std::max(d, F), qd)),
           ALR_E_UNSUPPORTED;
  if (wmax >= lim32)
    return fmt_msg(msg, len, "a weight matrix of the config is >= 4 GiB in bf16"),
           ALR_E_UNSUPPORTED;
  // the attention kernels copy key/value tiles by 32-bit byte offsets into one
  // layer's cache (tokens, or transposed-V columns with per-sequence padding)
  const double vt_cols = std::ceil((lim.max_tokens + 64.0 * lim.max_seqs) / 64.0) * 64.0;
  if (std::max((double)lim.max_tokens, vt_cols) * kvd * 2.0 >= lim32)
    return fmt_msg(msg, len, "one layer's key/value cache is >= 4 GiB (lower max_tokens)"),
           ALR_E_UNSUPPORTED;
  return ALR_OK;
}

int anchor_group(const alr_config& c) { return std::max(1, 128 / (c.n_heads / c.n_kv_heads)); }

bool mfma_attn(const alr_config& c) {
  return c.dtype == ALR_BF16 && (c.head_dim == 64 || c.head_dim == 128);
}

size_t compute_layout(const alr_config& c, const alr_limits& lim, Layout& L) {
  const size_t es = (c.dtype == ALR_BF16) ? 2 : 4;
  const size_t d = c.d_model, F = c.d_ffn, V = c.vocab, H = c.n_heads, G = c.n_kv_heads,
               hd = c.head_dim, nl = c.n_layers;
  const size_t qd = H * hd, kvd = G * hd;
  const size_t T = lim.max_tokens, NA = lim.max_anchors;
  const size_t R = std::max(T, NA);
  const size_t np = lim.max_block > 1 ? (size_t)(lim.max_block - 1) : 0;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  L.es = es;
  L.w_embed = take(V * d * es);
  L.w_lm = take(V * d * es);
  L.w_fnorm = take(d * es);
  {
    size_t lo = 0;
    auto ltake = [&](size_t bytes) {
      const size_t o = lo;
      lo = align256(lo + bytes);
      return o;
    };
    L.l_anorm = ltake(d * es);
    L.l_fnorm = ltake(d * es);
    L.l_qkv = ltake((qd + 2 * kvd) * d * es);
    L.l_o = ltake(d * qd * es);
    L.l_gu = ltake(2 * F * d * es);
    L.l_down = ltake(d * F * es);
    L.layer_stride = lo;
  }
  L.layer0 = take(nl * L.layer_stride);
  L.rope_cos = take((size_t)c.max_pos * (hd / 2) * 4);
  L.rope_sin = take((size_t)c.max_pos * (hd / 2) * 4);
  // transposed V (MFMA attention): [G*hd][vt_stride] per layer, every sequence
  // starting at a multiple of 64 columns
  L.vt_stride = mfma_attn(c) ? ((T + 64 * (size_t)lim.max_seqs + 63) / 64) * 64 : 0;
  L.kv_layer_stride = align256(std::max(T, L.vt_stride) * kvd * es);
  L.kc = take(nl * L.kv_layer_stride);
  L.vc = take(nl * L.kv_layer_stride);
  L.kvp_layer_stride = align256(NA * np * kvd * es);
  L.kp = take(nl * L.kvp_layer_stride);
  L.vp = take(nl * L.kvp_layer_stride);
  L.feat_store = take(T * (size_t)c.n_feat * d * 4);
  L.hf_store = take(T * d * es);
  L.resid = take(R * d * 4);
  L.xnorm = take(R * d * es);
  L.qbuf = take(R * qd * es);
  L.attn = take(R * qd * es);
  L.act = take(R * F * es);
  L.i_tokpos = take(T * 3 * 4);
  L.i_rowstart = take(T * 4);
  L.i_perm = take(NA * 4);
  L.i_apos = take(NA * 4);
  L.i_rpos = take(NA * 3 * 4);
  L.i_atok = take(NA * 4);
  L.i_aseq = take(NA * 4);
  L.i_alen = take(NA * 4);
  L.i_cur = take(NA * 4);
  L.i_valid = take(NA);
  L.i_target = take(NA * 4);
  L.i_ira = take(NA * 2 * 4);
  L.i_ctok = take(T * 4);
  L.logits = take(NA * V * 4);
  // output-head partials: one LogitPart per (anchor row, 64-column group)
  L.lm_part = take(NA * (V / 64) * sizeof(LogitPart));
  L.max_pwork = ((T + 31) / 32 + lim.max_seqs) * H + (size_t)lim.max_seqs * G;
  const size_t ag = (size_t)anchor_group(c);
  L.max_groups = (NA + ag - 1) / ag + std::min<size_t>(lim.max_seqs, NA);
  // chunks of >= ceil(total tiles / AT_DECODE_MAX_ITEMS) tiles: at most AT_DECODE_MAX_ITEMS
  // full chunks plus one partial chunk per (group, kv head), plus padding to a multiple of 8
  L.max_dwork = mfma_attn(c) ? AT_DECODE_MAX_ITEMS + L.max_groups * G + 8 : 0;
  L.i_pwork = take(L.max_pwork * sizeof(PrefillItem));
  L.i_dwork = take(L.max_dwork * sizeof(DecodeItem));
  L.i_maps = take(((qd + 2 * kvd) + 2 * F) * 4);
  L.i_rowptr = take(std::max((size_t)c.vocab, qd + 2 * kvd + 2 * d + 2 * F) * sizeof(void*));
  L.i_vtcol = take(T * 4);
  L.i_vtpad = take((size_t)lim.max_seqs * 2 * 4);
  L.i_rowinfo = take(NA * 2 * 4);
  L.part_o = take(L.max_dwork * 128 * hd * 2);  // fp16, normalised by the chunk sum
  L.part_ml = take(L.max_dwork * 128 * 2 * 4);
  // split-K partial sums of the rollout GEMMs: up to 4 slices of [anchors, N] fp32
  L.splitk_bytes = 4 * NA * std::max(qd + 2 * kvd, d) * 4;
  L.splitk = take(L.splitk_bytes);
  L.total = off;
  return off;
}

alr_status check_rollout_impl(const alr_config& c, const alr_limits& lim, int n_seq,
                              const int32_t* seq_len, int32_t n_anchor, const int32_t* aseq,
                              const int32_t* apos, int32_t block, char* msg, size_t len) {
  if (n_anchor <= 0 || n_anchor > lim.max_anchors)
    return fmt_msg(msg, len, "n_anchor %d outside [1, %d]", n_anchor, lim.max_anchors),
           ALR_E_INVALID_ARG;
  if (block <= 0 || block > lim.max_block)
    return fmt_msg(msg, len, "block %d outside [1, %d]", block, lim.max_block), ALR_E_INVALID_ARG;
  if (!aseq || !apos || !seq_len)
    return fmt_msg(msg, len, "anchor arrays must not be NULL"), ALR_E_INVALID_ARG;
  for (int i = 0; i < n_anchor; ++i) {
    if (aseq[i] < 0 || aseq[i] >= n_seq)
      return fmt_msg(msg, len, "anchor %d: sequence %d outside [0, %d)", i, aseq[i], n_seq),
             ALR_E_OUT_OF_RANGE;
    if (apos[i] < 0 || apos[i] >= seq_len[aseq[i]])
      return fmt_msg(msg, len, "anchor %d: position %d outside [0, %d)", i, apos[i],
                     seq_len[aseq[i]]),
             ALR_E_OUT_OF_RANGE;
    if ((long)apos[i] + block - 1 >= c.max_pos)
      return fmt_msg(msg, len, "anchor %d: last slot position %ld >= max_pos %d", i,
                     (long)apos[i] + block - 1, c.max_pos),
             ALR_E_OUT_OF_RANGE;
  }
  return ALR_OK;
}

alr_status check_prefill_impl(const alr_config& c, const alr_limits& lim, int32_t n_seq,
                              const int32_t* seq_len, const int32_t* tokens, const void* embeds,
                              const uint8_t* mask, char* msg, size_t len) {
  if (n_seq <= 0 || n_seq > lim.max_seqs)
    return fmt_msg(msg, len, "n_seq %d outside [1, %d]", n_seq, lim.max_seqs), ALR_E_INVALID_ARG;
  if (!seq_len || !tokens) return fmt_msg(msg, len, "seq_len and tokens must not be NULL"), ALR_E_INVALID_ARG;
  if ((embeds == nullptr) != (mask == nullptr))
    return fmt_msg(msg, len, "embeds and embed_mask must both be given or both be NULL"),
           ALR_E_INVALID_ARG;
  long tot = 0;
  for (int i = 0; i < n_seq; ++i) {
    if (seq_len[i] <= 0 || seq_len[i] > c.max_pos)
      return fmt_msg(msg, len, "seq_len[%d] = %d outside [1, max_pos=%d]", i, seq_len[i], c.max_pos),
             ALR_E_OUT_OF_RANGE;
    tot += seq_len[i];
  }
  if (tot > lim.max_tokens)
    return fmt_msg(msg, len, "total tokens %ld > max_tokens %d", tot, lim.max_tokens),
           ALR_E_OUT_OF_RANGE;
  return ALR_OK;
}

}  // namespace

struct alr_ctx {
  alr_config cfg;
  alr_limits lim;
  char* ws;
  size_t ws_bytes;
  Layout L;
  bool prefilled = false;
  int n_cu = 256;  // compute units of the device (sizes the decode work split)
  float* splitk_buf = nullptr;  // split-K partial sums (workspace)
  char* noalloc_scratch = nullptr;  // device address of `scratch` on the context's device
  std::string noalloc_err;          // why it could not be looked up, if it could not
  size_t splitk_bytes = 0;
  int n_seq = 0;
  std::vector<int> seq_len, seq_off;
  std::vector<int> h_tokpos, h_rowstart, h_vtcol, seq_vcol, h_vtpad;
  std::vector<PrefillItem> h_pwork;
  std::vector<int> h_anch;  // perm | apos | atok | aseq | alen (n each) | rope positions (3n)
  std::vector<int> h_ira;   // secondary primaries | offsets
  std::vector<DecodeItem> h_dwork;
  std::vector<DecodeGroup> h_groups;
  std::vector<int> h_grprow, h_rowinfo;
  std::string err;
  // launch timing of one site (alr_profile_*)
  int prof_site = 0;
  std::vector<hipEvent_t> prof_ev;
  size_t prof_used = 0;
  // rollout launch graphs (alr_set_rollout_graphs): the instantiated graphs,
  // least recently used first, and the private stream they are recorded and
  // replayed on, ordered after and before the caller's stream by two events
  struct RolloutGraph {
    std::array<uintptr_t, 12> key;
    hipGraphExec_t exec;
  };
  bool graphs_on = false;
  std::vector<RolloutGraph> graphs;
  hipStream_t graph_stream = nullptr;
  hipEvent_t graph_in = nullptr, graph_out = nullptr;

  template <typename P> P* at(size_t off) const { return reinterpret_cast<P*>(ws + off); }
  char* layer(int l) const { return ws + L.layer0 + (size_t)l * L.layer_stride; }
};

// Scratch of alr_rollout_topk_noalloc (each step's logit rows and their
// per-group partials), for callers that cannot allocate device memory.  Every
// device the library runs on holds its own copy until the process ends.  In
// host code this name is only a handle for hipGetSymbolAddress: kernels get the
// device address that call returns (noalloc_scratch_address).
static __device__ __align__(256) char scratch[ALR_NOALLOC_SCRATCH_BYTES];

namespace {

std::mutex g_scratch_mu;
std::vector<char*> g_scratch_addr;  // per device ordinal, looked up once

// Device address of `scratch` on the current device.
hipError_t noalloc_scratch_address(char** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if ((int)g_scratch_addr.size() <= dev) g_scratch_addr.resize(dev + 1, nullptr);
  if (g_scratch_addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_addr[dev] = static_cast<char*>(p);
  }
  *out = g_scratch_addr[dev];
  return hipSuccess;
}

alr_status fail(alr_ctx* ctx, alr_status st, const char* f, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, f);
  vsnprintf(buf, sizeof(buf), f, ap);
  va_end(ap);
  if (ctx) ctx->err = buf;
  else g_create_err = buf;
  return st;
}

#define ALR_HIP(ctx, call)                                                                 \
  do {                                                                                     \
    hipError_t e_ = (call);                                                                \
    if (e_ != hipSuccess)                                                                  \
      return fail(ctx, ALR_E_HIP, "%s failed: %s", #call, hipGetErrorString(e_));          \
  } while (0)

#define ALR_LAUNCHED(ctx, what)                                                            \
  do {                                                                                     \
    hipError_t e_ = hipGetLastError();                                                     \
    if (e_ != hipSuccess)                                                                  \
      return fail(ctx, ALR_E_HIP, "launch of %s failed: %s", what, hipGetErrorString(e_)); \
  } while (0)

// Event pair around one launch when `site` is the profiled one.
struct ProfScope {
  alr_ctx* ctx;
  hipStream_t st;
  hipEvent_t end = nullptr;
  ProfScope(alr_ctx* c, int site, hipStream_t s) : ctx(c), st(s) {
    if (c->prof_site == site && 2 * (c->prof_used + 1) <= c->prof_ev.size()) {
      (void)hipEventRecord(c->prof_ev[2 * c->prof_used], s);
      end = c->prof_ev[2 * c->prof_used + 1];
      ++c->prof_used;
    }
  }
  ~ProfScope() {
    if (end) (void)hipEventRecord(end, st);
  }
};

// Sum of the S fp32 K-slice partials of an M x N product, then the real
// epilogue; the slice counts the planner picks (2, 4) get kernels that load
// every partial before the first add.
template <class Epi>
void launch_splitk_reduce(const float* part, long sstride, int S, int M, int N, const Epi& epi,
                          hipStream_t st) {
  if constexpr (has_quad<Epi>::value) {
    const long thr4 = (long)M * (N / 64) * 8;
    const unsigned nb4 = (unsigned)((thr4 + 255) / 256);
    if (S == 2) {
      splitk_reduce4_kernel<Epi, 2><<<nb4, 256, 0, st>>>(part, sstride, M, N, epi);
      return;
    }
    if (S == 4) {
      splitk_reduce4_kernel<Epi, 4><<<nb4, 256, 0, st>>>(part, sstride, M, N, epi);
      return;
    }
  }
  const long thr = (long)M * (N / 64) * 32;
  const unsigned nb = (unsigned)((thr + 255) / 256);
  if (S == 2)
    splitk_reduce_kernel<Epi, 2><<<nb, 256, 0, st>>>(part, sstride, S, M, N, epi);
  else if (S == 4)
    splitk_reduce_kernel<Epi, 4><<<nb, 256, 0, st>>>(part, sstride, S, M, N, epi);
  else
    splitk_reduce_kernel<Epi, 0><<<nb, 256, 0, st>>>(part, sstride, S, M, N, epi);
}

// The split-K reduce of a residual update together with the RMSNorm that reads
// the updated rows (gains g, output out), when the row fits the fused kernel:
// one launch instead of two, bit-identical to them.  false leaves both to the
// caller.
template <typename T>
bool launch_splitk_resid_norm(alr_ctx* ctx, int S, int M, int N, const EpiResid& er, const T* g,
                              T* out, hipStream_t st) {
  if (er.ld != N || N % 4 != 0 || N > 8192 || (S != 2 && S != 4)) return false;
  const int ch = (N + 1023) / 1024;
  const float eps = ctx->cfg.rms_eps;
  const float* part = ctx->splitk_buf;
  const long ss = (long)M * N;
#define ALR_RN(S_, CH_)                                                                     \
  splitk_resid_norm_kernel<T, S_, CH_><<<M, 256, 0, st>>>(part, ss, er.h, er.feat, er.feat_rs, \
                                                          er.perm, g, out, N, eps)
  if (S == 2) {
    if (ch <= 1) ALR_RN(2, 1); else if (ch <= 2) ALR_RN(2, 2); else if (ch <= 4) ALR_RN(2, 4); else ALR_RN(2, 8);
  } else {
    if (ch <= 1) ALR_RN(4, 1); else if (ch <= 2) ALR_RN(4, 2); else if (ch <= 4) ALR_RN(4, 4); else ALR_RN(4, 8);
  }
#undef ALR_RN
  return true;
}

// norm_g / norm_out / normed: the RMSNorm that follows a residual update
// (Epi = EpiResid).  When the product takes a split-K path, it is fused into
// the reduce and *normed is set; otherwise the caller runs it.
template <int TAG, typename T, class Epi>
void launch_gemm(alr_ctx* ctx, const T* A, int lda, const T* W, int ldw, int M, int N, int K,
                 Epi epi, hipStream_t st, int force_tile = 0, const T* norm_g = nullptr,
                 T* norm_out = nullptr, bool* normed = nullptr) {
  if (M <= 0) return;
  ProfScope ps(ctx, TAG, st);
  if constexpr (std::is_same<T, bf16>::value) {
    // W row-major.  256x256 ping-pong (BK = 64), persistent over the tiles, for
    // the prefill and wide decode GEMMs, 128x128 (then 64x128) LDS-staged tiles
    // where 256x256 would leave CUs idle.  force_tile (debug hook only) picks any variant.
    auto tiles = [&](int bm, int bn) { return ((M + bm - 1) / bm) * ((N + bn - 1) / bn); };
    int cfg = force_tile;
    // Split-K over the 256x256 ping-pong kernel when its tiles leave CUs idle:
    // the largest slice count in {2, 4} that keeps one workgroup per CU, K
    // slices of >= 512 and a multiple of 64, and the partial sums in the buffer.
    // Where 128x128 tiles alone give every CU the same number of tiles and
    // K <= 4096, writing and re-reading the fp32 partial sums costs more than
    // the ping-pong kernel gains (M = 1024, N = 4096: 46 vs 55 us), so those
    // GEMMs take the 128x128 kernel with the epilogue fused (also where the
    // split-K reduce would carry the following RMSNorm: 29.5 vs 26.3 + 2.9 ms
    // per step for the rollout O projection).  With uneven rounds (N = 6144:
    // 384 tiles on 256 CUs) split-K stays ahead.
    const bool fill128 = K <= 4096 && tiles(128, 128) % ctx->n_cu == 0;
    // the output head's per-group partials are formed in the epilogue of each
    // tile; a split-K reduce hands it columns in another arrangement
    bool epi_whole_k = false;
    if constexpr (std::is_same<Epi, EpiLogits>::value) epi_whole_k = epi.part != nullptr;
    // Few rows (the rollout of a small batch): when even split-K leaves more
    // than half the CUs without a 256x256 tile, 64x128 tiles split over K
    // (slices of >= 256 and a multiple of 64) spread the work over more CUs.
    if ((cfg == 20 || (cfg == 0 && !fill128)) && ctx->splitk_buf != nullptr && !epi_whole_k) {
      const int t256 = tiles(256, 256), t64 = tiles(64, 128);
      int S256 = 1, S = 1;
      for (int cand : {2, 4}) {
        const bool fits = (size_t)cand * M * N * 4 <= ctx->splitk_bytes;
        if ((long)t256 * cand <= ctx->n_cu && K % (64 * cand) == 0 && K / cand >= 512 && fits)
          S256 = cand;
        if ((long)t64 * cand <= ctx->n_cu && K % (64 * cand) == 0 &&
            (K / cand >= 256 || cfg == 20) && fits)
          S = cand;
      }
      if (S > 1 && (cfg == 20 || ((long)t256 * S256 < ctx->n_cu / 2 && t64 * S >= 2 * t256 * S256))) {
        const int tm = (M + 63) / 64, tn = (N + 127) / 128;
        EpiPartial ep{ctx->splitk_buf, (long)M * N, N};
        if ((K / S) % 128 == 0)
          gemm_bf16_kernel<TAG, 64, 128, 2, 2, 64, 2, EpiPartial>
              <<<t64 * S, 256, 0, st>>>(A, lda, W, ldw, M, N, K / S, tm, tn, ep, S);
        else
          gemm_bf16_kernel<TAG, 64, 128, 2, 2, 32, 4, EpiPartial>
              <<<t64 * S, 256, 0, st>>>(A, lda, W, ldw, M, N, K / S, tm, tn, ep, S);
        if constexpr (std::is_same<Epi, EpiResid>::value) {
          if (norm_out && normed && launch_splitk_resid_norm<T>(ctx, S, M, N, epi, norm_g, norm_out, st)) {
            *normed = true;
            return;
          }
        }
        launch_splitk_reduce(ctx->splitk_buf, (long)M * N, S, M, N, epi, st);
        return;
      }
      if (cfg == 20) cfg = 3;
    }
    if ((cfg == 18 || (cfg == 0 && !fill128)) && ctx->splitk_buf != nullptr && !epi_whole_k) {
      const int t256 = tiles(256, 256);
      int S = 1;
      for (int cand : {2, 4})
        if ((long)t256 * cand <= ctx->n_cu && K % (64 * cand) == 0 && K / cand >= 512 &&
            (size_t)cand * M * N * 4 <= ctx->splitk_bytes)
          S = cand;
      if (cfg == 18 && S == 1 && K % 128 == 0 && (size_t)2 * M * N * 4 <= ctx->splitk_bytes) S = 2;
      if (S > 1 && (cfg == 18 || t256 < ctx->n_cu)) {
        const int tm = (M + 255) / 256, tn = (N + 255) / 256;
        EpiPartial ep{ctx->splitk_buf, (long)M * N, N};
        gemm_bf16_pp64_kernel<TAG, EpiPartial>
            <<<t256 * S, 512, 0, st>>>(A, lda, W, ldw, M, N, K / S, tm, tn, ep, S);
        if constexpr (std::is_same<Epi, EpiResid>::value) {
          if (norm_out && normed && launch_splitk_resid_norm<T>(ctx, S, M, N, epi, norm_g, norm_out, st)) {
            *normed = true;
            return;
          }
        }
        launch_splitk_reduce(ctx->splitk_buf, (long)M * N, S, M, N, epi, st);
        return;
      }
      if (cfg == 18) cfg = 0;
    }
    if (cfg == 0)
      cfg = tiles(256, 256) >= 256 ? ((K % 64) == 0 ? 19 : 4) : (tiles(128, 128) >= 256 ? 2 : 3);
    if ((cfg == 17 || cfg == 19) && (K % 64) != 0) cfg = 4;
    const bool k64 = (K % 128) == 0;
    const int bm = (cfg == 1 || cfg == 4 || cfg == 5 || cfg >= 17) ? 256 : (cfg == 3 ? 64 : 128);
    const int bn = (cfg == 4 || cfg == 5 || cfg >= 17) ? 256 : 128;
    const int tm = (M + bm - 1) / bm, tn = (N + bn - 1) / bn;
    const int nb = tm * tn;
#define ALR_GEMM(BM_, BN_, WGM_, WGN_, BK_, OCC_)                                      \
  gemm_bf16_kernel<TAG, BM_, BN_, WGM_, WGN_, BK_, OCC_, Epi>                          \
      <<<nb, 64 * WGM_ * WGN_, 0, st>>>(A, lda, W, ldw, M, N, K, tm, tn, epi)
    switch (cfg) {
      case 17:
        gemm_bf16_pp64_kernel<TAG, Epi><<<nb, 512, 0, st>>>(A, lda, W, ldw, M, N, K, tm, tn, epi);
        break;
      case 19:
        gemm_bf16_pp64p_kernel<TAG, Epi>
            <<<std::min(nb, ctx->n_cu), 512, 0, st>>>(A, lda, W, ldw, M, N, K, tm, tn, epi);
        break;
      case 5: if (k64) ALR_GEMM(256, 256, 2, 2, 64, 1); else ALR_GEMM(256, 256, 2, 2, 32, 1); break;
      case 4: if (k64) ALR_GEMM(256, 256, 2, 4, 64, 1); else ALR_GEMM(256, 256, 2, 4, 32, 1); break;
      case 1: if (k64) ALR_GEMM(256, 128, 2, 2, 64, 1); else ALR_GEMM(256, 128, 2, 2, 32, 1); break;
      case 2: if (k64) ALR_GEMM(128, 128, 2, 2, 64, 2); else ALR_GEMM(128, 128, 2, 2, 32, 2); break;
      default: if (k64) ALR_GEMM(64, 128, 2, 2, 64, 2); else ALR_GEMM(64, 128, 2, 2, 32, 4); break;
    }
#undef ALR_GEMM
  } else {
    const int tm = (M + GF_M - 1) / GF_M, tn = (N + GF_N - 1) / GF_N;
    gemm_f32_kernel<TAG, Epi><<<tm * tn, 256, 0, st>>>(A, lda, W, ldw, M, N, K, tm, tn, epi);
  }
}

AttnGeom geom(const alr_config& c) {
  AttnGeom g;
  g.H = c.n_heads;
  g.G = c.n_kv_heads;
  g.hd = c.head_dim;
  g.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)c.head_dim));
  return g;
}

// Column arrangement of the fused QKV weight: for q (n heads of hd), the
// original row feeding fused row (64 t + w) -- see EpiQKV.
void rope_pair_rows(int n, int hd, std::vector<int>& dst_of_src) {
  const int half = hd / 2, tot = n * hd;
  dst_of_src.assign(tot, -1);
  for (int nr = 0; nr < tot; ++nr) {
    const int t = nr / 64, w = nr % 64;
    const int f = 32 * t + (w & 31);
    const int head = f / half, i = f % half;
    const int src = head * hd + i + (w >= 32 ? half : 0);
    dst_of_src[src] = nr;
  }
}

// normed_in: the layer's input norm was already applied (fused into the
// previous layer's down-projection reduce).  next_g / next_out: the RMSNorm
// after this layer (the next layer's input norm or the final norm), which the
// down projection fuses into its reduce when it takes a split-K path; then
// *next_done is set.
template <typename T>
alr_status layer_forward(alr_ctx* ctx, int l, int M, bool decode, int s, float* feat,
                         long feat_rs, const int* perm, bool normed_in, const T* next_g,
                         T* next_out, bool* next_done, hipStream_t st) {
  const alr_config& c = ctx->cfg;
  const Layout& L = ctx->L;
  const int d = c.d_model, F = c.d_ffn, H = c.n_heads, G = c.n_kv_heads, hd = c.head_dim;
  const int qd = H * hd, kvd = G * hd;
  char* lw = ctx->layer(l);
  float* resid = ctx->at<float>(L.resid);
  T* xn = ctx->at<T>(L.xnorm);
  T* qb = ctx->at<T>(L.qbuf);
  T* at = ctx->at<T>(L.attn);
  T* act = ctx->at<T>(L.act);
  T* kc = reinterpret_cast<T*>(ctx->ws + L.kc + (size_t)l * L.kv_layer_stride);
  T* vc = reinterpret_cast<T*>(ctx->ws + L.vc + (size_t)l * L.kv_layer_stride);
  T* kp = reinterpret_cast<T*>(ctx->ws + L.kp + (size_t)l * L.kvp_layer_stride);
  T* vp = reinterpret_cast<T*>(ctx->ws + L.vp + (size_t)l * L.kvp_layer_stride);
  const int np = ctx->lim.max_block - 1;
  const long priv_rs = (long)np * kvd;

  if (!normed_in)
    rmsnorm_kernel<T><<<M, 256, 0, st>>>(resid, reinterpret_cast<const T*>(lw + L.l_anorm), xn, d,
                                         c.rms_eps);
  EpiQKV<T> eq;
  eq.q = qb;
  eq.cosT = ctx->at<float>(L.rope_cos);
  eq.sinT = ctx->at<float>(L.rope_sin);
  eq.H = H;
  eq.G = G;
  eq.hd = hd;
  {
    const int* ms = c.mrope_sections;
    const bool none = ms[0] == 0 && ms[1] == 0 && ms[2] == 0;
    eq.sec0 = none ? hd / 2 : ms[0];
    eq.sec01 = none ? hd / 2 : ms[0] + ms[1];
  }
  eq.vt_col = nullptr;
  eq.vt_stride = 0;
  if (!decode) {
    eq.k = kc;
    eq.v = vc;
    eq.kv_rs = kvd;
    eq.pos = ctx->at<int>(L.i_tokpos);
    eq.pos_add = 0;
    if (L.vt_stride) {
      eq.vt_col = ctx->at<int>(L.i_vtcol);
      eq.vt_stride = (long)L.vt_stride;
    }
  } else {
    eq.k = kp + (long)(s - 1) * kvd;
    eq.v = vp + (long)(s - 1) * kvd;
    eq.kv_rs = priv_rs;
    eq.pos = ctx->at<int>(L.i_rpos);
    eq.pos_add = s;
  }
  if (decode)
    launch_gemm<ALR_PROF_DECODE_QKV, T>(ctx, xn, d, reinterpret_cast<const T*>(lw + L.l_qkv), d, M,
                                        qd + 2 * kvd, d, eq, st);
  else
    launch_gemm<ALR_PROF_PREFILL_QKV, T>(ctx, xn, d, reinterpret_cast<const T*>(lw + L.l_qkv), d,
                                         M, qd + 2 * kvd, d, eq, st);
  ALR_LAUNCHED(ctx, "qkv gemm");

  const AttnGeom g = geom(c);
  {
  ProfScope ps(ctx, decode ? ALR_PROF_DECODE_ATTN : ALR_PROF_PREFILL_ATTN, st);
  if (!decode) {
    if (mfma_attn(c)) {
      const int nw = (int)ctx->h_pwork.size();
      const PrefillItem* wk = ctx->at<PrefillItem>(L.i_pwork);
      if constexpr (std::is_same<T, bf16>::value) {
        if (hd == 128)
          attn_prefill_mfma_kernel<128>
              <<<nw, 256, 0, st>>>(qb, kc, vc, (long)L.vt_stride, at, wk, g);
        else
          attn_prefill_mfma_kernel<64>
              <<<nw, 256, 0, st>>>(qb, kc, vc, (long)L.vt_stride, at, wk, g);
      }
    } else {
      const long items = (long)M * H;
      attn_generic_kernel<T><<<(unsigned)((items + 3) / 4), 256, 0, st>>>(
          qb, kc, vc, nullptr, nullptr, 0, 0, ctx->at<int>(L.i_rowstart), nullptr, at, M, g);
    }
  } else {
    if (mfma_attn(c)) {
      const int nw = (int)ctx->h_dwork.size();
      const DecodeItem* wk = ctx->at<DecodeItem>(L.i_dwork);
      uint16_t* po = ctx->at<uint16_t>(L.part_o);
      float* pml = ctx->at<float>(L.part_ml);
      const unsigned ncomb = (unsigned)(((long)M * G + 3) / 4);
      const int2* rinfo = ctx->at<int2>(L.i_rowinfo);
      if constexpr (std::is_same<T, bf16>::value) {
        if (hd == 128) {
          attn_decode_mfma_kernel<128><<<nw, 256, 0, st>>>(qb, kc, vc, (long)L.vt_stride,
                                                            ctx->at<int>(L.i_apos), wk, po, pml, g);
          ProfScope pc(ctx, ALR_PROF_DECODE_COMBINE, st);
          attn_decode_combine_kernel<128><<<ncomb, 256, 0, st>>>(rinfo, po, pml, qb, kp, vp,
                                                                 priv_rs, s, at, M, g);
        } else {
          attn_decode_mfma_kernel<64><<<nw, 256, 0, st>>>(qb, kc, vc, (long)L.vt_stride,
                                                           ctx->at<int>(L.i_apos), wk, po, pml, g);
          ProfScope pc(ctx, ALR_PROF_DECODE_COMBINE, st);
          attn_decode_combine_kernel<64><<<ncomb, 256, 0, st>>>(rinfo, po, pml, qb, kp, vp,
                                                                priv_rs, s, at, M, g);
        }
      }
    } else {
      const long items = (long)M * H;
      attn_generic_kernel<T><<<(unsigned)((items + 3) / 4), 256, 0, st>>>(
          qb, kc, vc, kp, vp, priv_rs, s, ctx->at<int>(L.i_aseq), ctx->at<int>(L.i_apos), at, M,
          g);
    }
  }
  }
  ALR_LAUNCHED(ctx, "attention");

  EpiResid er;
  er.h = resid;
  er.ld = d;
  er.feat = nullptr;
  er.feat_rs = 0;
  er.perm = nullptr;
  const T* fnorm = reinterpret_cast<const T*>(lw + L.l_fnorm);
  bool fnormed = false;
  if (decode)
    launch_gemm<ALR_PROF_DECODE_O, T>(ctx, at, qd, reinterpret_cast<const T*>(lw + L.l_o), qd, M,
                                      d, qd, er, st, 0, fnorm, xn, &fnormed);
  else
    launch_gemm<ALR_PROF_PREFILL_O, T>(ctx, at, qd, reinterpret_cast<const T*>(lw + L.l_o), qd, M,
                                       d, qd, er, st, 0, fnorm, xn, &fnormed);
  if (!fnormed)
    rmsnorm_kernel<T><<<M, 256, 0, st>>>(resid, fnorm, xn, d, c.rms_eps);
  EpiSwiGLU<T> es;
  es.out = act;
  es.ld = F;
  if (decode)
    launch_gemm<ALR_PROF_DECODE_GU, T>(ctx, xn, d, reinterpret_cast<const T*>(lw + L.l_gu), d, M,
                                       2 * F, d, es, st);
  else
    launch_gemm<ALR_PROF_PREFILL_GU, T>(ctx, xn, d, reinterpret_cast<const T*>(lw + L.l_gu), d, M,
                                        2 * F, d, es, st);
  er.feat = feat;
  er.feat_rs = feat_rs;
  er.perm = perm;
  *next_done = false;
  if (decode)
    launch_gemm<ALR_PROF_DECODE_DOWN, T>(ctx, act, F, reinterpret_cast<const T*>(lw + L.l_down), F,
                                         M, d, F, er, st, 0, next_g, next_out, next_done);
  else
    launch_gemm<ALR_PROF_PREFILL_DOWN, T>(ctx, act, F, reinterpret_cast<const T*>(lw + L.l_down),
                                          F, M, d, F, er, st, 0, next_g, next_out, next_done);
  ALR_LAUNCHED(ctx, "mlp");
  return ALR_OK;
}

int feat_index(const alr_config& c, int l) {
  for (int f = 0; f < c.n_feat; ++f)
    if (c.feat_layers[f] == l) return f;
  return -1;
}

template <typename T>
alr_status prefill_impl(alr_ctx* ctx, int M, const int32_t* tokens, const void* embeds,
                        const uint8_t* mask, float* feats_out, hipStream_t st) {
  const alr_config& c = ctx->cfg;
  const Layout& L = ctx->L;
  const int d = c.d_model, nf = c.n_feat;
  embed_kernel<T><<<M, 256, 0, st>>>(ctx->at<float>(L.resid), tokens, ctx->at<T>(L.w_embed),
                                     reinterpret_cast<const T*>(embeds), mask, d);
  keep_tokens_kernel<<<(M + 255) / 256, 256, 0, st>>>(ctx->at<int>(L.i_ctok), tokens, mask, M);
  ALR_LAUNCHED(ctx, "embed");
  if constexpr (std::is_same<T, bf16>::value) {
    bool any_pad = false;
    for (int i = 0; i < ctx->n_seq; ++i) any_pad |= ctx->h_vtpad[2 * i + 1] > 0;
    if (L.vt_stride && any_pad && c.n_layers > 0) {
      const int rows = c.n_kv_heads * c.head_dim;
      const long total = (long)c.n_layers * rows * ctx->n_seq;
      zero_vt_pad_kernel<<<(unsigned)((total + 255) / 256), 256, 0, st>>>(
          reinterpret_cast<bf16*>(ctx->ws + L.vc), (long)(L.kv_layer_stride / 2),
          (long)L.vt_stride, ctx->at<int>(L.i_vtpad), ctx->n_seq, rows, total);
      ALR_LAUNCHED(ctx, "transposed-V padding");
    }
  }
  bool normed = false;  // the next layer's input norm (or the final norm) already applied
  for (int l = 0; l < c.n_layers; ++l) {
    const int f = feat_index(c, l);
    float* feat = f >= 0 ? ctx->at<float>(L.feat_store) + (long)f * d : nullptr;
    const bool last = l + 1 == c.n_layers;
    const T* ng = last ? ctx->at<T>(L.w_fnorm)
                       : reinterpret_cast<const T*>(ctx->layer(l + 1) + L.l_anorm);
    T* no = last ? ctx->at<T>(L.hf_store) : ctx->at<T>(L.xnorm);
    bool done = false;
    const alr_status stt = layer_forward<T>(ctx, l, M, false, 0, feat, (long)nf * d, nullptr,
                                            normed, ng, no, &done, st);
    if (stt != ALR_OK) return stt;
    normed = done;
  }
  if (!normed)
    rmsnorm_kernel<T><<<M, 256, 0, st>>>(ctx->at<float>(L.resid), ctx->at<T>(L.w_fnorm),
                                         ctx->at<T>(L.hf_store), d, c.rms_eps);
  ALR_LAUNCHED(ctx, "final norm");
  if (feats_out && nf > 0)
    ALR_HIP(ctx, hipMemcpyAsync(feats_out, ctx->at<float>(L.feat_store),
                                (size_t)M * nf * d * sizeof(float), hipMemcpyDeviceToDevice, st));
  return ALR_OK;
}

// Output destinations of the labels of one rollout or corpus-label call.
struct LabelDst {
  float* logprobs;  // [n, block, V] or null (then the logits go to the logit rows below)
  int* tokens;      // argmax per slot [n, block]
  int* top_ids;     // [n, block, 8] or null (no top-8 labels)
  float* top_logp;
  float* tail;
  float* logit_rows = nullptr;      // [n, V] scratch for the logits; null: the workspace's
  LogitPart* part_rows = nullptr;   // [n, V/64] scratch for the partials; null: the workspace's
};

// Output head of slot s for the n sorted rows in xnorm: logits GEMM (into the
// caller's log-prob rows, or the workspace rows when none are wanted), then
// the finalisation.  `rollout` feeds the next tokens (forced or greedy);
// otherwise the rows' validity and corpus targets come from the workspace.
template <typename T>
alr_status lm_head(alr_ctx* ctx, int n, int s, int block, const int* forced, const LabelDst& out,
                   bool rollout, float* target_logp, hipStream_t st) {
  const alr_config& c = ctx->cfg;
  const Layout& L = ctx->L;
  const int V = c.vocab, d = c.d_model;
  const int* perm = ctx->at<int>(L.i_perm);
  EpiLogits el;
  LmFinalize f;
  el.part = out.part_rows ? out.part_rows : ctx->at<LogitPart>(L.lm_part);
  el.part_ld = V / 64;
  f.part = el.part;
  f.part_ld = el.part_ld;
  if (out.logprobs) {
    el.out = out.logprobs + (long)s * V;
    el.rs = (long)block * V;
    el.perm = perm;
    f.z = out.logprobs + (long)s * V;
    f.z_rs = (long)block * V;
    f.z_perm = 1;
    f.write_lp = 1;
  } else {
    float* rows = out.logit_rows ? out.logit_rows : ctx->at<float>(L.logits);
    el.out = rows;
    el.rs = V;
    el.perm = nullptr;
    f.z = rows;
    f.z_rs = V;
    f.z_perm = 0;
    f.write_lp = 0;
  }
  launch_gemm<ALR_PROF_LM_GEMM, T>(ctx, ctx->at<T>(L.xnorm), d, ctx->at<T>(L.w_lm), d, n, V, d,
                                   el, st);
  f.perm = perm;
  f.V = V;
  f.block = block;
  f.s = s;
  f.tokens = out.tokens;
  f.forced = rollout ? forced : nullptr;
  f.next_tok = rollout ? ctx->at<int>(L.i_cur) : nullptr;
  f.top_ids = out.top_ids;
  f.top_logp = out.top_logp;
  f.tail = out.tail;
  f.target = rollout ? nullptr : ctx->at<int>(L.i_target);
  f.target_logp = rollout ? nullptr : target_logp;
  f.valid = rollout ? nullptr : ctx->at<unsigned char>(L.i_valid);
  {
    ProfScope ps(ctx, ALR_PROF_LM_FINALIZE, st);
    if (out.top_ids)
      lm_finalize_kernel<true><<<n, 256, 0, st>>>(f);
    else
      lm_finalize_kernel<false><<<n, 256, 0, st>>>(f);
  }
  ALR_LAUNCHED(ctx, "output head");
  return ALR_OK;
}

template <typename T>
alr_status rollout_impl(alr_ctx* ctx, int n, int block, const int32_t* forced, const LabelDst& out,
                        float* feats_out, hipStream_t st) {
  const alr_config& c = ctx->cfg;
  const Layout& L = ctx->L;
  const int d = c.d_model, nf = c.n_feat;
  const int* perm = ctx->at<int>(L.i_perm);
  const int* atok = ctx->at<int>(L.i_atok);
  // slot 0: the prefill's final-norm row and features at the anchor
  gather_rows_kernel<T><<<n, 256, 0, st>>>(ctx->at<T>(L.xnorm), ctx->at<T>(L.hf_store), atok, d);
  if (feats_out && nf > 0)
    gather_feat_kernel<<<n, 256, 0, st>>>(feats_out, (long)block * nf * d, perm,
                                          ctx->at<float>(L.feat_store), atok, (long)nf * d);
  ALR_LAUNCHED(ctx, "slot-0 gather");
  alr_status stt = lm_head<T>(ctx, n, 0, block, forced, out, true, nullptr, st);
  if (stt != ALR_OK) return stt;
  for (int s = 1; s < block; ++s) {
    embed_kernel<T><<<n, 256, 0, st>>>(ctx->at<float>(L.resid), ctx->at<int>(L.i_cur),
                                       ctx->at<T>(L.w_embed), nullptr, nullptr, d);
    ALR_LAUNCHED(ctx, "decode embed");
    bool normed = false;  // as in the prefill
    for (int l = 0; l < c.n_layers; ++l) {
      const int f = feat_index(c, l);
      float* feat = (f >= 0 && feats_out) ? feats_out + ((long)s * nf + f) * d : nullptr;
      const T* ng = l + 1 == c.n_layers
                        ? ctx->at<T>(L.w_fnorm)
                        : reinterpret_cast<const T*>(ctx->layer(l + 1) + L.l_anorm);
      bool done = false;
      stt = layer_forward<T>(ctx, l, n, true, s, feat, (long)block * nf * d, perm, normed, ng,
                             ctx->at<T>(L.xnorm), &done, st);
      if (stt != ALR_OK) return stt;
      normed = done;
    }
    if (!normed)
      rmsnorm_kernel<T><<<n, 256, 0, st>>>(ctx->at<float>(L.resid), ctx->at<T>(L.w_fnorm),
                                           ctx->at<T>(L.xnorm), d, c.rms_eps);
    stt = lm_head<T>(ctx, n, s, block, forced, out, true, nullptr, st);
    if (stt != ALR_OK) return stt;
  }
  return ALR_OK;
}

constexpr size_t kMaxRolloutGraphs = 4;

// The graphs run on the context's own stream: waiting for it first means no
// graph is destroyed while a launch of it may still execute.
void drop_rollout_graphs(alr_ctx* ctx) {
  if (ctx->graphs.empty()) return;
  (void)hipStreamSynchronize(ctx->graph_stream);
  for (auto& g : ctx->graphs) (void)hipGraphExecDestroy(g.exec);
  ctx->graphs.clear();
}

// rollout_impl through a cached HIP graph.  Besides the context's constants,
// the launches of one rollout depend only on the key below (anchor count,
// block, the size of the attention work list, the output and input pointers):
// anchors, positions and plans reach the kernels through the workspace and are
// uploaded on the caller's stream before the graph runs, so a graph recorded
// for one call replays every later call with the same key.  The graph is
// recorded and run on the context's own stream (the null stream cannot be
// captured), which waits for the caller's stream and which the caller's stream
// then waits for.  Plain launches while a launch site of the rollout is being
// timed (its event pairs are recorded per launch), when the caller's stream is
// itself being captured, or when graphs are off.
template <typename T>
alr_status run_rollout(alr_ctx* ctx, int n, int block, const int32_t* forced, const LabelDst& out,
                       float* feats_out, hipStream_t st, bool allow_graph) {
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  const bool timing_rollout_site = ctx->prof_site >= ALR_PROF_DECODE_QKV;
  if (!allow_graph || !ctx->graphs_on || timing_rollout_site || n <= 0)
    return rollout_impl<T>(ctx, n, block, forced, out, feats_out, st);
  ALR_HIP(ctx, hipStreamIsCapturing(st, &cap));
  if (cap != hipStreamCaptureStatusNone)
    return rollout_impl<T>(ctx, n, block, forced, out, feats_out, st);
  hipStream_t gs = ctx->graph_stream;  // created by alr_set_rollout_graphs
  const std::array<uintptr_t, 12> key{
      (uintptr_t)n, (uintptr_t)block, (uintptr_t)ctx->h_dwork.size(), (uintptr_t)forced,
      (uintptr_t)feats_out, (uintptr_t)out.logprobs, (uintptr_t)out.tokens,
      (uintptr_t)out.top_ids, (uintptr_t)out.top_logp, (uintptr_t)out.tail,
      (uintptr_t)out.logit_rows, (uintptr_t)out.part_rows};
  ALR_HIP(ctx, hipEventRecord(ctx->graph_in, st));
  ALR_HIP(ctx, hipStreamWaitEvent(gs, ctx->graph_in, 0));
  hipGraphExec_t exec = nullptr;
  for (size_t i = 0; i < ctx->graphs.size(); ++i) {
    if (ctx->graphs[i].key == key) {
      const alr_ctx::RolloutGraph g = ctx->graphs[i];
      ctx->graphs.erase(ctx->graphs.begin() + (long)i);
      ctx->graphs.push_back(g);
      exec = g.exec;
      break;
    }
  }
  if (!exec) {
    ALR_HIP(ctx, hipStreamBeginCapture(gs, hipStreamCaptureModeThreadLocal));
    const alr_status rs = rollout_impl<T>(ctx, n, block, forced, out, feats_out, gs);
    hipGraph_t graph = nullptr;
    const hipError_t ec = hipStreamEndCapture(gs, &graph);
    if (rs != ALR_OK || ec != hipSuccess || !graph) {
      if (graph) (void)hipGraphDestroy(graph);
      if (rs != ALR_OK) return rs;
      return fail(ctx, ALR_E_HIP, "rollout graph capture failed: %s", hipGetErrorString(ec));
    }
    const hipError_t ei = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    if (ei != hipSuccess)
      return fail(ctx, ALR_E_HIP, "rollout graph instantiation failed: %s", hipGetErrorString(ei));
    if (ctx->graphs.size() >= kMaxRolloutGraphs) {
      // the least recently used graph may be the last one launched on gs
      ALR_HIP(ctx, hipStreamSynchronize(gs));
      (void)hipGraphExecDestroy(ctx->graphs.front().exec);
      ctx->graphs.erase(ctx->graphs.begin());
    }
    ctx->graphs.push_back({key, exec});
  }
  ALR_HIP(ctx, hipGraphLaunch(exec, gs));
  ALR_HIP(ctx, hipEventRecord(ctx->graph_out, gs));
  ALR_HIP(ctx, hipStreamWaitEvent(st, ctx->graph_out, 0));
  return ALR_OK;
}

// Corpus labels: for every slot s, the prefill's final-norm rows at a + s
// through the output head, the corpus token's log-prob, then the gates.
template <typename T>
alr_status corpus_impl(alr_ctx* ctx, int n, int block, const LabelDst& out, float* corpus_logp,
                       float* gate_soft, float* gate_hard, hipStream_t st) {
  const alr_config& c = ctx->cfg;
  const Layout& L = ctx->L;
  const int d = c.d_model;
  for (int s = 0; s < block; ++s) {
    corpus_rows_kernel<T><<<n, 256, 0, st>>>(
        ctx->at<T>(L.xnorm), ctx->at<T>(L.hf_store), ctx->at<int>(L.i_atok),
        ctx->at<int>(L.i_apos), ctx->at<int>(L.i_alen), ctx->at<int>(L.i_ctok), s, d,
        ctx->at<unsigned char>(L.i_valid), ctx->at<int>(L.i_target));
    ALR_LAUNCHED(ctx, "corpus rows");
    const alr_status stt = lm_head<T>(ctx, n, s, block, nullptr, out, false, corpus_logp, st);
    if (stt != ALR_OK) return stt;
  }
  erase_gates_kernel<<<(n + 255) / 256, 256, 0, st>>>(
      ctx->at<int>(L.i_perm), ctx->at<int>(L.i_atok), ctx->at<int>(L.i_apos),
      ctx->at<int>(L.i_alen), ctx->at<int>(L.i_ctok), corpus_logp, out.tokens, n, block,
      gate_soft, gate_hard);
  ALR_LAUNCHED(ctx, "erase gates");
  return ALR_OK;
}

alr_status upload(alr_ctx* ctx, void* dst, const void* src, size_t bytes, hipStream_t st) {
  if (bytes == 0) return ALR_OK;
  ALR_HIP(ctx, hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, st));
  return ALR_OK;
}

}  // namespace

// ============================================================== C ABI

extern "C" {

const char* alr_status_string(alr_status st) {
  switch (st) {
    case ALR_OK: return "ALR_OK";
    case ALR_E_INVALID_ARG: return "ALR_E_INVALID_ARG";
    case ALR_E_OUT_OF_RANGE: return "ALR_E_OUT_OF_RANGE";
    case ALR_E_WORKSPACE: return "ALR_E_WORKSPACE";
    case ALR_E_STATE: return "ALR_E_STATE";
    case ALR_E_UNSUPPORTED: return "ALR_E_UNSUPPORTED";
    case ALR_E_HIP: return "ALR_E_HIP";
  }
  return "unknown status";
}

alr_status alr_check_config(const alr_config* cfg, char* msg, size_t msg_len) {
  return check_config_impl(cfg, msg, msg_len);
}

size_t alr_workspace_bytes(const alr_config* cfg, const alr_limits* lim) {
  if (check_config_impl(cfg, nullptr, 0) != ALR_OK || check_limits(lim, nullptr, 0) != ALR_OK ||
      check_operand_sizes(*cfg, *lim, nullptr, 0) != ALR_OK)
    return 0;
  Layout L;
  return compute_layout(*cfg, *lim, L);
}

alr_status alr_check_rollout(const alr_config* cfg, const alr_limits* lim, int32_t n_seq,
                             const int32_t* seq_len, int32_t n_anchor, const int32_t* anchor_seq,
                             const int32_t* anchor_pos, int32_t block, char* msg, size_t msg_len) {
  alr_status st = check_config_impl(cfg, msg, msg_len);
  if (st != ALR_OK) return st;
  st = check_limits(lim, msg, msg_len);
  if (st != ALR_OK) return st;
  if (n_seq <= 0 || n_seq > lim->max_seqs)
    return fmt_msg(msg, msg_len, "n_seq %d outside [1, %d]", n_seq, lim->max_seqs),
           ALR_E_INVALID_ARG;
  return check_rollout_impl(*cfg, *lim, n_seq, seq_len, n_anchor, anchor_seq, anchor_pos, block,
                            msg, msg_len);
}

alr_status alr_create(const alr_config* cfg, const alr_weights* w, const alr_limits* lim,
                      void* workspace, size_t ws_bytes, alr_stream stream, alr_ctx** out) {
  char msg[256];
  if (!out) return fail(nullptr, ALR_E_INVALID_ARG, "out is NULL");
  *out = nullptr;
  alr_status st = check_config_impl(cfg, msg, sizeof(msg));
  if (st != ALR_OK) return fail(nullptr, st, "%s", msg);
  st = check_limits(lim, msg, sizeof(msg));
  if (st != ALR_OK) return fail(nullptr, st, "%s", msg);
  st = check_operand_sizes(*cfg, *lim, msg, sizeof(msg));
  if (st != ALR_OK) return fail(nullptr, st, "%s", msg);
  const alr_config& c = *cfg;
  if (!w || !w->tok_embed || !w->final_norm || !w->lm_head)
    return fail(nullptr, ALR_E_INVALID_ARG, "weights: tok_embed, final_norm and lm_head required");
  if (c.n_layers > 0 && (!w->attn_norm || !w->wq || !w->wk || !w->wv || !w->wo || !w->ffn_norm ||
                         !w->w_gate || !w->w_up || !w->w_down))
    return fail(nullptr, ALR_E_INVALID_ARG, "weights: per-layer pointer arrays required");
  for (int l = 0; l < c.n_layers; ++l)
    if (!w->attn_norm[l] || !w->wq[l] || !w->wk[l] || !w->wv[l] || !w->wo[l] || !w->ffn_norm[l] ||
        !w->w_gate[l] || !w->w_up[l] || !w->w_down[l])
      return fail(nullptr, ALR_E_INVALID_ARG, "weights of layer %d incomplete", l);
  Layout L;
  const size_t need = compute_layout(c, *lim, L);
  if (!workspace) return fail(nullptr, ALR_E_INVALID_ARG, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % 256)
    return fail(nullptr, ALR_E_INVALID_ARG, "workspace must be 256-byte aligned");
  if (ws_bytes < need)
    return fail(nullptr, ALR_E_WORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, need);

  alr_ctx* ctx = new alr_ctx();
  ctx->cfg = c;
  ctx->lim = *lim;
  ctx->ws = static_cast<char*>(workspace);
  ctx->ws_bytes = ws_bytes;
  ctx->L = L;
  hipStream_t s = static_cast<hipStream_t>(stream);
  auto bad = [&](alr_status e) {
    g_create_err = ctx->err;
    delete ctx;
    return e;
  };
#define CREATE_HIP(call)                                                             \
  do {                                                                               \
    hipError_t e_ = (call);                                                          \
    if (e_ != hipSuccess) {                                                          \
      fail(ctx, ALR_E_HIP, "%s failed: %s", #call, hipGetErrorString(e_));           \
      return bad(ALR_E_HIP);                                                         \
    }                                                                                \
  } while (0)

  {
    int dev = 0, ncu = 0;
    CREATE_HIP(hipGetDevice(&dev));
    CREATE_HIP(hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev));
    ctx->n_cu = std::max(1, ncu);
  }
  {
    // with the context's device current: the no-alloc entry point's scratch
    const hipError_t e = noalloc_scratch_address(&ctx->noalloc_scratch);
    if (e != hipSuccess) {
      ctx->noalloc_scratch = nullptr;
      ctx->noalloc_err = hipGetErrorString(e);
      (void)hipGetLastError();
    }
  }
  ctx->splitk_buf = ctx->at<float>(L.splitk);
  ctx->splitk_bytes = L.splitk_bytes;
  const size_t es = L.es, d = c.d_model, F = c.d_ffn, V = c.vocab;
  const int H = c.n_heads, G = c.n_kv_heads, hd = c.head_dim;
  const size_t qd = (size_t)H * hd, kvd = (size_t)G * hd;
  CREATE_HIP(hipMemcpyAsync(ctx->ws + L.w_embed, w->tok_embed, V * d * es, hipMemcpyDeviceToDevice, s));
  CREATE_HIP(hipMemcpyAsync(ctx->ws + L.w_fnorm, w->final_norm, d * es, hipMemcpyDeviceToDevice, s));

  // Fused weight rows: q and k rows are arranged so that every rotate-half
  // partner sits 32 columns after its pair (rope_pair_rows), gate and up rows
  // alternate in blocks of 32.  src_of[n] is the source row of fused row n.
  std::vector<int> qmap, kmap;
  rope_pair_rows(H, hd, qmap);
  rope_pair_rows(G, hd, kmap);
  std::vector<int> q_src(qd), k_src(kvd);
  for (size_t i = 0; i < qd; ++i) q_src[qmap[i]] = (int)i;
  for (size_t i = 0; i < kvd; ++i) k_src[kmap[i]] = (int)i;
  if (c.dtype == ALR_BF16) {
    // bf16: fused weights assembled row-major from a table of source rows
    const size_t qkv = qd + 2 * kvd;
    std::vector<const bf16*> rp;
    const void** drp = ctx->at<const void*>(L.i_rowptr);
    auto shuffle = [&](char* dst, const bf16* const* rows_dev, int N, int K) {
      const long chunks = (long)N * (K / 8);
      gather_rows_ptr_kernel<<<(unsigned)((chunks + 255) / 256), 256, 0, s>>>(
          reinterpret_cast<bf16*>(dst), rows_dev, N, K);
    };
    rp.resize(V);
    for (size_t n = 0; n < V; ++n) rp[n] = (const bf16*)w->lm_head + n * d;
    CREATE_HIP(hipMemcpyAsync(drp, rp.data(), V * sizeof(void*), hipMemcpyHostToDevice, s));
    shuffle(ctx->ws + L.w_lm, (const bf16* const*)drp, (int)V, (int)d);
    CREATE_HIP(hipGetLastError());
    CREATE_HIP(hipStreamSynchronize(s));  // the pointer table is rewritten below
    for (int l = 0; l < c.n_layers; ++l) {
      char* lw = ctx->layer(l);
      CREATE_HIP(hipMemcpyAsync(lw + L.l_anorm, w->attn_norm[l], d * es, hipMemcpyDeviceToDevice, s));
      CREATE_HIP(hipMemcpyAsync(lw + L.l_fnorm, w->ffn_norm[l], d * es, hipMemcpyDeviceToDevice, s));
      rp.clear();
      for (size_t n = 0; n < qd; ++n) rp.push_back((const bf16*)w->wq[l] + (size_t)q_src[n] * d);
      for (size_t n = 0; n < kvd; ++n) rp.push_back((const bf16*)w->wk[l] + (size_t)k_src[n] * d);
      for (size_t n = 0; n < kvd; ++n) rp.push_back((const bf16*)w->wv[l] + n * d);
      for (size_t n = 0; n < d; ++n) rp.push_back((const bf16*)w->wo[l] + n * qd);
      for (size_t n = 0; n < 2 * F; ++n) {
        const size_t t = n / 64, wi = n % 64;
        rp.push_back(wi < 32 ? (const bf16*)w->w_gate[l] + (t * 32 + wi) * d
                             : (const bf16*)w->w_up[l] + (t * 32 + wi - 32) * d);
      }
      for (size_t n = 0; n < d; ++n) rp.push_back((const bf16*)w->w_down[l] + n * F);
      CREATE_HIP(hipMemcpyAsync(drp, rp.data(), rp.size() * sizeof(void*), hipMemcpyHostToDevice, s));
      const bf16* const* r0 = (const bf16* const*)drp;
      shuffle(lw + L.l_qkv, r0, (int)qkv, (int)d);
      shuffle(lw + L.l_o, r0 + qkv, (int)d, (int)qd);
      shuffle(lw + L.l_gu, r0 + qkv + d, (int)(2 * F), (int)d);
      shuffle(lw + L.l_down, r0 + qkv + d + 2 * F, (int)d, (int)F);
      CREATE_HIP(hipGetLastError());
      CREATE_HIP(hipStreamSynchronize(s));
    }
  } else {
    CREATE_HIP(hipMemcpyAsync(ctx->ws + L.w_lm, w->lm_head, V * d * es, hipMemcpyDeviceToDevice, s));
    std::vector<int> maps;  // destination row of each source row
    maps.reserve(qd + 2 * kvd + 2 * F);
    for (int x : qmap) maps.push_back(x);
    for (int x : kmap) maps.push_back((int)qd + x);
    for (size_t i = 0; i < kvd; ++i) maps.push_back((int)(qd + kvd + i));
    for (size_t i = 0; i < F; ++i) maps.push_back((int)((i / 32) * 64 + (i % 32)));       // gate
    for (size_t i = 0; i < F; ++i) maps.push_back((int)((i / 32) * 64 + 32 + (i % 32)));  // up
    int* dmaps = ctx->at<int>(L.i_maps);
    CREATE_HIP(hipMemcpyAsync(dmaps, maps.data(), maps.size() * 4, hipMemcpyHostToDevice, s));
    const long rb = (long)d * es;
    for (int l = 0; l < c.n_layers; ++l) {
      char* lw = ctx->layer(l);
      CREATE_HIP(hipMemcpyAsync(lw + L.l_anorm, w->attn_norm[l], d * es, hipMemcpyDeviceToDevice, s));
      CREATE_HIP(hipMemcpyAsync(lw + L.l_fnorm, w->ffn_norm[l], d * es, hipMemcpyDeviceToDevice, s));
      scatter_rows_kernel<<<(unsigned)qd, 256, 0, s>>>(lw + L.l_qkv, (const char*)w->wq[l], dmaps, rb);
      scatter_rows_kernel<<<(unsigned)kvd, 256, 0, s>>>(lw + L.l_qkv, (const char*)w->wk[l],
                                                        dmaps + qd, rb);
      scatter_rows_kernel<<<(unsigned)kvd, 256, 0, s>>>(lw + L.l_qkv, (const char*)w->wv[l],
                                                        dmaps + qd + kvd, rb);
      CREATE_HIP(hipMemcpyAsync(lw + L.l_o, w->wo[l], d * qd * es, hipMemcpyDeviceToDevice, s));
      scatter_rows_kernel<<<(unsigned)F, 256, 0, s>>>(lw + L.l_gu, (const char*)w->w_gate[l],
                                                      dmaps + qd + 2 * kvd, rb);
      scatter_rows_kernel<<<(unsigned)F, 256, 0, s>>>(lw + L.l_gu, (const char*)w->w_up[l],
                                                      dmaps + qd + 2 * kvd + F, rb);
      CREATE_HIP(hipMemcpyAsync(lw + L.l_down, w->w_down[l], d * F * es, hipMemcpyDeviceToDevice, s));
      CREATE_HIP(hipGetLastError());
    }
  }
  // RoPE tables: angles in double, stored as float cos/sin [max_pos, hd/2]
  {
    const int half = hd / 2;
    std::vector<float> cs((size_t)c.max_pos * half), sn((size_t)c.max_pos * half);
    for (int i = 0; i < half; ++i) {
      const double inv = std::pow((double)c.rope_base, -2.0 * i / hd);
      for (int p = 0; p < c.max_pos; ++p) {
        const double a = p * inv;
        cs[(size_t)p * half + i] = (float)std::cos(a);
        sn[(size_t)p * half + i] = (float)std::sin(a);
      }
    }
    CREATE_HIP(hipMemcpyAsync(ctx->ws + L.rope_cos, cs.data(), cs.size() * 4, hipMemcpyHostToDevice, s));
    CREATE_HIP(hipMemcpyAsync(ctx->ws + L.rope_sin, sn.data(), sn.size() * 4, hipMemcpyHostToDevice, s));
    CREATE_HIP(hipStreamSynchronize(s));
  }
#undef CREATE_HIP
  *out = ctx;
  return ALR_OK;
}

alr_status alr_prefill(alr_ctx* ctx, int32_t n_seq, const int32_t* seq_len, const int32_t* tokens,
                       const void* embeds, const uint8_t* embed_mask, float* feats_out,
                       alr_stream stream) {
  return alr_prefill_positions(ctx, n_seq, seq_len, tokens, nullptr, embeds, embed_mask, feats_out,
                               stream);
}

alr_status alr_prefill_positions(alr_ctx* ctx, int32_t n_seq, const int32_t* seq_len,
                                 const int32_t* tokens, const int32_t* positions,
                                 const void* embeds, const uint8_t* embed_mask, float* feats_out,
                                 alr_stream stream) {
  if (!ctx) return ALR_E_INVALID_ARG;
  char msg[256];
  alr_status st = check_prefill_impl(ctx->cfg, ctx->lim, n_seq, seq_len, tokens, embeds,
                                     embed_mask, msg, sizeof(msg));
  if (st != ALR_OK) return fail(ctx, st, "%s", msg);
  if (positions) {
    long tot = 0;
    for (int i = 0; i < n_seq; ++i) tot += seq_len[i];
    for (long t = 0; t < 3 * tot; ++t)
      if (positions[t] < 0 || positions[t] >= ctx->cfg.max_pos)
        return fail(ctx, ALR_E_OUT_OF_RANGE, "positions[%ld][%ld] = %d outside [0, max_pos=%d)",
                    t / 3, t % 3, positions[t], ctx->cfg.max_pos);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const alr_config& c = ctx->cfg;
  const int rep = c.n_heads / c.n_kv_heads;
  ctx->prefilled = false;
  ctx->n_seq = n_seq;
  ctx->seq_len.assign(seq_len, seq_len + n_seq);
  ctx->seq_off.assign(n_seq + 1, 0);
  for (int i = 0; i < n_seq; ++i) ctx->seq_off[i + 1] = ctx->seq_off[i] + seq_len[i];
  const int M = ctx->seq_off[n_seq];
  ctx->h_tokpos.resize((size_t)3 * M);
  ctx->h_rowstart.resize(M);
  ctx->h_pwork.clear();
  ctx->h_vtcol.resize(M);
  ctx->seq_vcol.assign(n_seq, 0);
  int vcol = 0;
  for (int i = 0; i < n_seq; ++i) {
    ctx->seq_vcol[i] = vcol;
    for (int p = 0; p < seq_len[i]; ++p) {
      const long row = ctx->seq_off[i] + p;
      for (int ax = 0; ax < 3; ++ax) ctx->h_tokpos[3 * row + ax] = positions ? positions[3 * row + ax] : p;
      ctx->h_rowstart[ctx->seq_off[i] + p] = ctx->seq_off[i];
      ctx->h_vtcol[ctx->seq_off[i] + p] = vcol + p;
    }
    vcol += (seq_len[i] + 63) / 64 * 64;
    const int n_items = ((seq_len[i] + 31) / 32) * rep;
    for (int g = 0; g < c.n_kv_heads; ++g)
      for (int it = 0; it < n_items; it += 4)
        ctx->h_pwork.push_back(PrefillItem{ctx->seq_off[i], ctx->seq_vcol[i], seq_len[i], g, it});
  }
  ctx->h_vtpad.assign((size_t)2 * n_seq, 0);
  for (int i = 0; i < n_seq; ++i) {
    ctx->h_vtpad[2 * i] = ctx->seq_vcol[i] + seq_len[i];
    ctx->h_vtpad[2 * i + 1] = (seq_len[i] + 63) / 64 * 64 - seq_len[i];
  }
  // causal work grows with the query position: start the longest items first
  std::stable_sort(ctx->h_pwork.begin(), ctx->h_pwork.end(),
                   [rep](const PrefillItem& a, const PrefillItem& b) {
                     return a.item0 / rep > b.item0 / rep;
                   });
  if (ctx->h_pwork.size() > ctx->L.max_pwork)
    return fail(ctx, ALR_E_WORKSPACE, "prefill work list overflow");
  const Layout& L = ctx->L;
  st = upload(ctx, ctx->at<int>(L.i_tokpos), ctx->h_tokpos.data(), (size_t)M * 3 * 4, s);
  if (st == ALR_OK) st = upload(ctx, ctx->at<int>(L.i_rowstart), ctx->h_rowstart.data(), (size_t)M * 4, s);
  if (st == ALR_OK) st = upload(ctx, ctx->at<int>(L.i_vtcol), ctx->h_vtcol.data(), (size_t)M * 4, s);
  if (st == ALR_OK)
    st = upload(ctx, ctx->at<int>(L.i_vtpad), ctx->h_vtpad.data(), (size_t)n_seq * 2 * 4, s);
  if (st == ALR_OK)
    st = upload(ctx, ctx->at<PrefillItem>(L.i_pwork), ctx->h_pwork.data(),
                ctx->h_pwork.size() * sizeof(PrefillItem), s);
  if (st != ALR_OK) return st;
  st = (c.dtype == ALR_BF16) ? prefill_impl<bf16>(ctx, M, tokens, embeds, embed_mask, feats_out, s)
                             : prefill_impl<float>(ctx, M, tokens, embeds, embed_mask, feats_out, s);
  if (st == ALR_OK) ctx->prefilled = true;
  return st;
}

namespace {

// Validates an anchor request, sorts the anchors by (sequence, position) and
// uploads the per-anchor tables (and, for a rollout, the decode-attention work
// split) to the workspace on stream s.
// Decode attention work plan for n anchors sorted by (sequence, position):
// seqs[r] and apos[r] are sorted anchor r's sequence and position; seq_off and
// seq_vcol give each sequence's first K-cache row and first V^T column.
// Fills the work items (dealt to XCDs: item b runs on XCD b % 8, padding
// items have count 0), the anchor groups and each sorted anchor's group.
// Returns the chunk length in 64-key tiles; *makespan receives the simulated
// makespan in tiles.
int plan_decode(const alr_config& c, int n_cu, int n, const int* seqs, const int* apos,
                const int* seq_off, const int* seq_vcol, std::vector<DecodeItem>& dwork,
                std::vector<DecodeGroup>& groups, std::vector<int>& grprow,
                long* makespan = nullptr) {
  dwork.clear();
  groups.clear();
  grprow.assign(n, 0);
  // Groups of up to 128/rep sorted anchors of one sequence.  The shared keys
  // 0..a_max of a group are cut, per kv head, into chunks of ct 64-key tiles
  // at absolute key positions, so the groups of one sequence read the same
  // chunks.  Work items are listed by (sequence, kv head, chunk, group) and
  // dealt in contiguous runs to the XCDs (workgroup b is dispatched to XCD
  // b % 8), so the groups sharing a chunk meet in that XCD's L2; within an
  // XCD the items go largest first (stable), so the short tail chunks fill
  // the slots the long ones leave.  ct minimises the makespan of that
  // order under list scheduling on the XCD's 2 * CUs / 8 workgroup slots,
  // an item costing its tiles + AT_DECODE_ITEM_OVERHEAD.
  const int ag = anchor_group(c), G = c.n_kv_heads;
  struct Grp {
    int f, cnt, sq, a_max, ntile;
  };
  std::vector<Grp> gs;
  long total_tiles = 0;
  for (int r0 = 0; r0 < n;) {
    const int sq = seqs[r0];
    int r1 = r0;
    while (r1 < n && seqs[r1] == sq) ++r1;
    for (int f = r0; f < r1; f += ag) {
      const int cnt = std::min(ag, r1 - f);
      const int a_max = apos[f + cnt - 1];
      gs.push_back(Grp{f, cnt, sq, a_max, (a_max + AT_KT) / AT_KT});
      total_tiles += (long)gs.back().ntile * G;
    }
    r0 = r1;
  }
  int max_nt = 1;
  for (const Grp& gr : gs) max_nt = std::max(max_nt, gr.ntile);
  const int ct_min = (int)std::max<long>(
      AT_DECODE_MIN_TILES, (total_tiles + AT_DECODE_MAX_ITEMS - 1) / AT_DECODE_MAX_ITEMS);
  // logical item list for chunk length ct: (group index, chunk)
  auto list_items = [&](int ct, std::vector<std::pair<int, int>>& out, std::vector<int>& kvh) {
    out.clear();
    kvh.clear();
    for (size_t g0 = 0; g0 < gs.size();) {  // g0..g1: the groups of one sequence
      size_t g1 = g0;
      int max_chunks = 0;
      while (g1 < gs.size() && gs[g1].sq == gs[g0].sq) {
        max_chunks = std::max(max_chunks, (gs[g1].ntile + ct - 1) / ct);
        ++g1;
      }
      for (int g = 0; g < G; ++g)
        for (int ch = 0; ch < max_chunks; ++ch)
          for (size_t gi = g0; gi < g1; ++gi)
            if (ch < (gs[gi].ntile + ct - 1) / ct) {
              out.emplace_back((int)gi, ch);
              kvh.push_back(g);
            }
      g0 = g1;
    }
  };
  auto item_tiles = [&](int ct, const std::pair<int, int>& it) {
    return std::min(ct, gs[it.first].ntile - it.second * ct);
  };
  // XCD x runs logical items [x * per, (x + 1) * per), largest first
  auto xcd_order = [&](int ct, const std::vector<std::pair<int, int>>& lg, size_t per, int x) {
    std::vector<int> idx;
    for (size_t li = (size_t)x * per; li < std::min(lg.size(), (size_t)(x + 1) * per); ++li)
      idx.push_back((int)li);
    std::stable_sort(idx.begin(), idx.end(), [&](int u, int v) {
      return item_tiles(ct, lg[u]) > item_tiles(ct, lg[v]);
    });
    return idx;
  };
  const int xslots = std::max(1, 2 * n_cu / 8);
  std::vector<std::pair<int, int>> lg;
  std::vector<int> lg_kvh;
  int ct = std::max(ct_min, max_nt);
  long best = -1;
  for (int cand = std::max(ct_min, max_nt); cand >= ct_min; --cand) {
    list_items(cand, lg, lg_kvh);
    const size_t per = (lg.size() + 7) / 8;
    long span = 0;
    for (int x = 0; x < 8; ++x) {
      // busy-until time of each slot; the next item goes to the earliest
      std::priority_queue<long, std::vector<long>, std::greater<long>> slot;
      for (int i = 0; i < xslots; ++i) slot.push(0);
      long last = 0;
      for (int li : xcd_order(cand, lg, per, x)) {
        const long t = slot.top() + item_tiles(cand, lg[li]) + AT_DECODE_ITEM_OVERHEAD;
        slot.pop();
        slot.push(t);
        last = std::max(last, t);
      }
      span = std::max(span, last);
    }
    if (best < 0 || span < best) {
      best = span;
      ct = cand;
    }
  }
  int part = 0;
  for (size_t gi = 0; gi < gs.size(); ++gi) {
    const int nchunk = (gs[gi].ntile + ct - 1) / ct;
    groups.push_back(DecodeGroup{gs[gi].f, nchunk, part});
    for (int rr = gs[gi].f; rr < gs[gi].f + gs[gi].cnt; ++rr) grprow[rr] = (int)gi;
    part += nchunk * G;
  }
  list_items(ct, lg, lg_kvh);
  const size_t per = (lg.size() + 7) / 8;
  dwork.assign(per * 8, DecodeItem{0, 0, 0, 0, 0, 0, 0, 0});
  for (int x = 0; x < 8; ++x) {
    const std::vector<int> idx = xcd_order(ct, lg, per, x);
    for (size_t i = 0; i < idx.size(); ++i) {
      const int gi = lg[idx[i]].first, ch = lg[idx[i]].second, g = lg_kvh[idx[i]];
      const DecodeGroup& dg = groups[gi];
      const int kb = ch * ct * AT_KT;
      const int ke = std::min(gs[gi].a_max + 1, kb + ct * AT_KT);
      dwork[x + 8 * i] = DecodeItem{gs[gi].f, gs[gi].cnt, g, seq_off[gs[gi].sq],
                                    seq_vcol[gs[gi].sq], kb, ke, dg.part0 + g * dg.nchunk + ch};
    }
  }
  if (makespan) *makespan = best;
  return ct;
}

alr_status prepare_anchors(alr_ctx* ctx, int32_t n_anchor, const int32_t* anchor_seq,
                           const int32_t* anchor_pos, int32_t block, bool rollout,
                           hipStream_t s) {
  if (!ctx->prefilled) return fail(ctx, ALR_E_STATE, "call before a successful prefill");
  char msg[256];
  alr_status st = check_rollout_impl(ctx->cfg, ctx->lim, ctx->n_seq, ctx->seq_len.data(), n_anchor,
                                     anchor_seq, anchor_pos, block, msg, sizeof(msg));
  if (st != ALR_OK) return fail(ctx, st, "%s", msg);
  const alr_config& c = ctx->cfg;
  const int n = n_anchor;
  std::vector<int> order(n);
  std::iota(order.begin(), order.end(), 0);
  std::sort(order.begin(), order.end(), [&](int x, int y) {
    if (anchor_seq[x] != anchor_seq[y]) return anchor_seq[x] < anchor_seq[y];
    if (anchor_pos[x] != anchor_pos[y]) return anchor_pos[x] < anchor_pos[y];
    return x < y;
  });
  ctx->h_anch.resize((size_t)8 * n);
  int* perm = ctx->h_anch.data();
  int* apos = perm + n;
  int* atok = perm + 2 * n;
  int* aseq = perm + 3 * n;
  int* alen = perm + 4 * n;
  int* rpos = perm + 5 * n;  // [n][3]: RoPE position of the anchor token on each axis
  for (int r = 0; r < n; ++r) {
    const int i = order[r];
    perm[r] = i;
    apos[r] = anchor_pos[i];
    atok[r] = ctx->seq_off[anchor_seq[i]] + anchor_pos[i];
    aseq[r] = ctx->seq_off[anchor_seq[i]];
    alen[r] = ctx->seq_len[anchor_seq[i]];
    for (int ax = 0; ax < 3; ++ax) {
      rpos[3 * r + ax] = ctx->h_tokpos[3 * (size_t)atok[r] + ax];
      if ((long)rpos[3 * r + ax] + block - 1 >= c.max_pos)
        return fail(ctx, ALR_E_OUT_OF_RANGE,
                    "anchor %d: position %d on axis %d + block - 1 >= max_pos %d", i,
                    rpos[3 * r + ax], ax, c.max_pos);
    }
  }
  ctx->h_dwork.clear();
  ctx->h_groups.clear();
  ctx->h_grprow.assign(n, 0);
  if (rollout) {
    if (mfma_attn(c)) {
      std::vector<int> sq_sorted(n);
      for (int r = 0; r < n; ++r) sq_sorted[r] = anchor_seq[order[r]];
      plan_decode(c, ctx->n_cu, n, sq_sorted.data(), apos, ctx->seq_off.data(),
                  ctx->seq_vcol.data(), ctx->h_dwork, ctx->h_groups, ctx->h_grprow);
    }
  }
  // per sorted row: its first partial row (kv head 0, chunk 0) and its group's chunk count
  ctx->h_rowinfo.assign((size_t)2 * n, 0);
  if (!ctx->h_groups.empty()) {
    const int rep_h = c.n_heads / c.n_kv_heads;
    for (int r = 0; r < n; ++r) {
      const DecodeGroup& dg = ctx->h_groups[ctx->h_grprow[r]];
      ctx->h_rowinfo[2 * r] = dg.part0 * 128 + (r - dg.first) * rep_h;
      ctx->h_rowinfo[2 * r + 1] = dg.nchunk;
    }
  }
  if (ctx->h_dwork.size() > ctx->L.max_dwork || ctx->h_groups.size() > ctx->L.max_groups)
    return fail(ctx, ALR_E_WORKSPACE, "decode work list overflow");
  const Layout& L = ctx->L;
  st = upload(ctx, ctx->at<int>(L.i_perm), perm, (size_t)n * 4, s);
  if (st == ALR_OK) st = upload(ctx, ctx->at<int>(L.i_apos), apos, (size_t)n * 4, s);
  if (st == ALR_OK) st = upload(ctx, ctx->at<int>(L.i_atok), atok, (size_t)n * 4, s);
  if (st == ALR_OK) st = upload(ctx, ctx->at<int>(L.i_aseq), aseq, (size_t)n * 4, s);
  if (st == ALR_OK) st = upload(ctx, ctx->at<int>(L.i_alen), alen, (size_t)n * 4, s);
  if (st == ALR_OK) st = upload(ctx, ctx->at<int>(L.i_rpos), rpos, (size_t)n * 3 * 4, s);
  if (st == ALR_OK && !ctx->h_dwork.empty())
    st = upload(ctx, ctx->at<DecodeItem>(L.i_dwork), ctx->h_dwork.data(),
                ctx->h_dwork.size() * sizeof(DecodeItem), s);

  if (st == ALR_OK && rollout)
    st = upload(ctx, ctx->at<int>(L.i_rowinfo), ctx->h_rowinfo.data(), (size_t)n * 2 * 4, s);
  return st;
}

}  // namespace

alr_status alr_rollout(alr_ctx* ctx, int32_t n_anchor, const int32_t* anchor_seq,
                       const int32_t* anchor_pos, int32_t block, const int32_t* forced,
                       int32_t* tokens_out, float* logprobs_out, float* feats_out,
                       alr_stream stream) {
  if (!ctx) return ALR_E_INVALID_ARG;
  if (!tokens_out || !logprobs_out)
    return fail(ctx, ALR_E_INVALID_ARG, "tokens_out and logprobs_out must not be NULL");
  hipStream_t s = static_cast<hipStream_t>(stream);
  alr_status st = prepare_anchors(ctx, n_anchor, anchor_seq, anchor_pos, block, true, s);
  if (st != ALR_OK) return st;
  const LabelDst out{logprobs_out, tokens_out, nullptr, nullptr, nullptr};
  return (ctx->cfg.dtype == ALR_BF16)
             ? run_rollout<bf16>(ctx, n_anchor, block, forced, out, feats_out, s, true)
             : run_rollout<float>(ctx, n_anchor, block, forced, out, feats_out, s, true);
}

alr_status alr_rollout_topk(alr_ctx* ctx, int32_t n_anchor, const int32_t* anchor_seq,
                            const int32_t* anchor_pos, int32_t block, const int32_t* forced,
                            int32_t* tokens_out, int32_t* top_ids_out, float* top_logp_out,
                            float* tail_out, float* logprobs_out, float* feats_out,
                            alr_stream stream) {
  if (!ctx) return ALR_E_INVALID_ARG;
  if (!tokens_out || !top_ids_out || !top_logp_out || !tail_out)
    return fail(ctx, ALR_E_INVALID_ARG,
                "tokens_out, top_ids_out, top_logp_out and tail_out must not be NULL");
  hipStream_t s = static_cast<hipStream_t>(stream);
  alr_status st = prepare_anchors(ctx, n_anchor, anchor_seq, anchor_pos, block, true, s);
  if (st != ALR_OK) return st;
  const LabelDst out{logprobs_out, tokens_out, top_ids_out, top_logp_out, tail_out};
  return (ctx->cfg.dtype == ALR_BF16)
             ? run_rollout<bf16>(ctx, n_anchor, block, forced, out, feats_out, s, true)
             : run_rollout<float>(ctx, n_anchor, block, forced, out, feats_out, s, true);
}

alr_status alr_rollout_topk_noalloc(alr_ctx* ctx, int32_t n_anchor, const int32_t* anchor_seq,
                                    const int32_t* anchor_pos, int32_t block,
                                    const int32_t* forced, int32_t* tokens_out,
                                    int32_t* top_ids_out, float* top_logp_out, float* tail_out,
                                    float* feats_out, alr_stream stream) {
  if (!ctx) return ALR_E_INVALID_ARG;
  if (!tokens_out || !top_ids_out || !top_logp_out || !tail_out)
    return fail(ctx, ALR_E_INVALID_ARG,
                "tokens_out, top_ids_out, top_logp_out and tail_out must not be NULL");
  const size_t V = (size_t)ctx->cfg.vocab;
  const size_t per_row = V * 4 + (V / 64) * sizeof(LogitPart);
  if (n_anchor > 0 && align256((size_t)n_anchor * V * 4) +
                          (size_t)n_anchor * (V / 64) * sizeof(LogitPart) >
                      (size_t)ALR_NOALLOC_SCRATCH_BYTES)
    return fail(ctx, ALR_E_WORKSPACE,
                "n_anchor %d needs %zu bytes of scratch at vocab %zu, more than the %zu-byte "
                "no-alloc scratch (at most %zu anchors)",
                n_anchor, (size_t)n_anchor * per_row, V, (size_t)ALR_NOALLOC_SCRATCH_BYTES,
                ((size_t)ALR_NOALLOC_SCRATCH_BYTES - 256) / per_row);
  if (!ctx->noalloc_scratch)
    return fail(ctx, ALR_E_HIP, "scratch address lookup failed at alr_create: %s",
                ctx->noalloc_err.c_str());
  hipStream_t s = static_cast<hipStream_t>(stream);
  alr_status st = prepare_anchors(ctx, n_anchor, anchor_seq, anchor_pos, block, true, s);
  if (st != ALR_OK) return st;
  LabelDst out{nullptr, tokens_out, top_ids_out, top_logp_out, tail_out};
  out.logit_rows = reinterpret_cast<float*>(ctx->noalloc_scratch);
  out.part_rows = reinterpret_cast<LogitPart*>(ctx->noalloc_scratch +
                                               align256((size_t)n_anchor * V * 4));
  return (ctx->cfg.dtype == ALR_BF16)
             ? rollout_impl<bf16>(ctx, n_anchor, block, forced, out, feats_out, s)
             : rollout_impl<float>(ctx, n_anchor, block, forced, out, feats_out, s);
}

alr_status alr_corpus_labels(alr_ctx* ctx, int32_t n_anchor, const int32_t* anchor_seq,
                             const int32_t* anchor_pos, int32_t block, int32_t* argmax_out,
                             int32_t* top_ids_out, float* top_logp_out, float* tail_out,
                             float* logprobs_out, float* corpus_logp_out, float* gate_soft_out,
                             float* gate_hard_out, alr_stream stream) {
  if (!ctx) return ALR_E_INVALID_ARG;
  if (!argmax_out || !corpus_logp_out || !gate_soft_out || !gate_hard_out)
    return fail(ctx, ALR_E_INVALID_ARG,
                "argmax_out, corpus_logp_out, gate_soft_out and gate_hard_out must not be NULL");
  if ((top_ids_out == nullptr) != (top_logp_out == nullptr) ||
      (top_ids_out == nullptr) != (tail_out == nullptr))
    return fail(ctx, ALR_E_INVALID_ARG,
                "top_ids_out, top_logp_out and tail_out must all be given or all be NULL");
  if (!top_ids_out && !logprobs_out)
    return fail(ctx, ALR_E_INVALID_ARG, "give top-8 outputs, log-prob rows or both");
  hipStream_t s = static_cast<hipStream_t>(stream);
  alr_status st = prepare_anchors(ctx, n_anchor, anchor_seq, anchor_pos, block, false, s);
  if (st != ALR_OK) return st;
  const LabelDst out{logprobs_out, argmax_out, top_ids_out, top_logp_out, tail_out};
  return (ctx->cfg.dtype == ALR_BF16)
             ? corpus_impl<bf16>(ctx, n_anchor, block, out, corpus_logp_out, gate_soft_out,
                                 gate_hard_out, s)
             : corpus_impl<float>(ctx, n_anchor, block, out, corpus_logp_out, gate_soft_out,
                                  gate_hard_out, s);
}

alr_status alr_ira_assemble(alr_ctx* ctx, int32_t n_primary, int32_t block,
                            const int32_t* tokens, const int32_t* top_ids, const float* top_logp,
                            const float* tail, int32_t n_secondary, const int32_t* sec_primary,
                            const int32_t* sec_offset, float gamma, int32_t eos_id,
                            int32_t* token0_out, int32_t* top_ids_out, float* top_logp_out,
                            float* tail_out, float* weight_out, alr_stream stream) {
  if (!ctx) return ALR_E_INVALID_ARG;
  if (n_primary <= 0 || n_primary > ctx->lim.max_anchors || block < 2 ||
      block > ctx->lim.max_block)
    return fail(ctx, ALR_E_INVALID_ARG, "n_primary %d / block %d outside the context limits",
                n_primary, block);
  if (n_secondary < 0 || n_secondary > ctx->lim.max_anchors)
    return fail(ctx, ALR_E_INVALID_ARG, "n_secondary %d outside [0, %d]", n_secondary,
                ctx->lim.max_anchors);
  if (!(gamma > 0.f)) return fail(ctx, ALR_E_INVALID_ARG, "gamma must be > 0");
  if (n_secondary == 0) return ALR_OK;
  if (!tokens || !top_ids || !top_logp || !tail || !sec_primary || !sec_offset || !token0_out ||
      !top_ids_out || !top_logp_out || !tail_out || !weight_out)
    return fail(ctx, ALR_E_INVALID_ARG, "NULL pointer argument");
  std::vector<int>& tab = ctx->h_ira;  // kept until the next call: the copy is asynchronous
  tab.assign((size_t)2 * n_secondary, 0);
  for (int q = 0; q < n_secondary; ++q) {
    if (sec_primary[q] < 0 || sec_primary[q] >= n_primary)
      return fail(ctx, ALR_E_OUT_OF_RANGE, "secondary %d: primary %d outside [0, %d)", q,
                  sec_primary[q], n_primary);
    if (sec_offset[q] < 1 || sec_offset[q] > block - 1)
      return fail(ctx, ALR_E_OUT_OF_RANGE, "secondary %d: offset %d outside [1, %d]", q,
                  sec_offset[q], block - 1);
    tab[q] = sec_primary[q];
    tab[n_secondary + q] = sec_offset[q];
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  int* dtab = ctx->at<int>(ctx->L.i_ira);
  const alr_status st = upload(ctx, dtab, tab.data(), tab.size() * 4, s);
  if (st != ALR_OK) return st;
  const long items = (long)n_secondary * block;
  ira_assemble_kernel<<<(unsigned)((items + 255) / 256), 256, 0, s>>>(
      dtab, dtab + n_secondary, n_secondary, block, tokens, top_ids, top_logp, tail, gamma,
      eos_id, token0_out, top_ids_out, top_logp_out, tail_out, weight_out);
  ALR_LAUNCHED(ctx, "in-rollout anchor assembly");
  return ALR_OK;
}

alr_status alr_slot_weights(alr_ctx* ctx, int32_t n, int32_t block, const int32_t* tokens,
                            int32_t eos_id, float gamma, float* weight_out, alr_stream stream) {
  if (!ctx) return ALR_E_INVALID_ARG;
  if (n < 0 || block < 1) return fail(ctx, ALR_E_INVALID_ARG, "n %d / block %d invalid", n, block);
  if (!(gamma > 0.f)) return fail(ctx, ALR_E_INVALID_ARG, "gamma must be > 0");
  if (n == 0) return ALR_OK;
  if (!tokens || !weight_out) return fail(ctx, ALR_E_INVALID_ARG, "NULL pointer argument");
  hipStream_t s = static_cast<hipStream_t>(stream);
  slot_weights_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(tokens, n, block, eos_id, gamma,
                                                                 weight_out);
  ALR_LAUNCHED(ctx, "slot weights");
  return ALR_OK;
}

const char* alr_last_error(const alr_ctx* ctx) {
  return ctx ? ctx->err.c_str() : g_create_err.c_str();
}

alr_status alr_set_rollout_graphs(alr_ctx* ctx, int32_t enable) {
  if (!ctx) return ALR_E_INVALID_ARG;
  if (enable != 0 && enable != 1)
    return fail(ctx, ALR_E_INVALID_ARG, "enable must be 0 or 1, got %d", enable);
  if (enable == 1 && !ctx->graph_stream) {  // the stream and its two events: all three or none
    hipStream_t gs0 = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    hipError_t e = hipStreamCreateWithFlags(&gs0, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&e0, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&e1, hipEventDisableTiming);
    if (e != hipSuccess) {
      if (e1) (void)hipEventDestroy(e1);
      if (e0) (void)hipEventDestroy(e0);
      if (gs0) (void)hipStreamDestroy(gs0);
      return fail(ctx, ALR_E_HIP, "rollout graph stream or events: %s", hipGetErrorString(e));
    }
    ctx->graph_stream = gs0;
    ctx->graph_in = e0;
    ctx->graph_out = e1;
  }
  ctx->graphs_on = enable == 1;
  if (!ctx->graphs_on) drop_rollout_graphs(ctx);
  return ALR_OK;
}

void alr_destroy(alr_ctx* ctx) {
  if (!ctx) return;
  for (hipEvent_t e : ctx->prof_ev) (void)hipEventDestroy(e);
  drop_rollout_graphs(ctx);
  if (ctx->graph_in) (void)hipEventDestroy(ctx->graph_in);
  if (ctx->graph_out) (void)hipEventDestroy(ctx->graph_out);
  if (ctx->graph_stream) (void)hipStreamDestroy(ctx->graph_stream);
  delete ctx;
}

// ------------------------------------------------------------------ debug hooks

alr_status alr_debug_decode_plan(const alr_config* cfg, int32_t n_cu, int32_t n_seq,
                                 const int32_t* seq_len, int32_t n_anchor,
                                 const int32_t* anchor_seq, const int32_t* anchor_pos,
                                 int32_t* ct_out, int32_t* makespan_out, int32_t* n_items_out,
                                 int32_t* items_out, int32_t max_items) {
  if (!cfg || !seq_len || !ct_out || !makespan_out || !n_items_out || n_seq <= 0 || n_cu <= 0)
    return ALR_E_INVALID_ARG;
  alr_status st = alr_check_config(cfg, nullptr, 0);
  if (st != ALR_OK) return st;
  if (!mfma_attn(*cfg)) return ALR_E_UNSUPPORTED;
  std::vector<int> off(n_seq + 1, 0), vcol(n_seq, 0);
  for (int i = 0; i < n_seq; ++i) {
    if (seq_len[i] <= 0) return ALR_E_INVALID_ARG;
    off[i + 1] = off[i] + seq_len[i];
    if (i + 1 < n_seq) vcol[i + 1] = vcol[i] + (seq_len[i] + 63) / 64 * 64;
  }
  const alr_limits lim{off[n_seq], n_seq, n_anchor, 1};
  st = check_rollout_impl(*cfg, lim, n_seq, seq_len, n_anchor, anchor_seq, anchor_pos, 1, nullptr,
                          0);
  if (st != ALR_OK) return st;
  const int n = n_anchor;
  std::vector<int> order(n);
  std::iota(order.begin(), order.end(), 0);
  std::sort(order.begin(), order.end(), [&](int x, int y) {
    if (anchor_seq[x] != anchor_seq[y]) return anchor_seq[x] < anchor_seq[y];
    if (anchor_pos[x] != anchor_pos[y]) return anchor_pos[x] < anchor_pos[y];
    return x < y;
  });
  std::vector<int> sq(n), ap(n);
  for (int r = 0; r < n; ++r) {
    sq[r] = anchor_seq[order[r]];
    ap[r] = anchor_pos[order[r]];
  }
  std::vector<DecodeItem> items;
  std::vector<DecodeGroup> groups;
  std::vector<int> grprow;
  long span = 0;
  *ct_out = plan_decode(*cfg, n_cu, n, sq.data(), ap.data(), off.data(), vcol.data(), items,
                        groups, grprow, &span);
  *makespan_out = (int32_t)span;
  *n_items_out = (int32_t)items.size();
  if (items_out) {
    if ((long)items.size() > max_items) return ALR_E_WORKSPACE;
    for (size_t b = 0; b < items.size(); ++b) {
      const DecodeItem& it = items[b];
      int32_t* o = items_out + 6 * b;
      o[0] = it.first;
      o[1] = it.count;
      o[2] = it.kvh;
      o[3] = it.kbeg;
      o[4] = it.kend;
      o[5] = it.part;
    }
  }
  return ALR_OK;
}

alr_status alr_debug_gemm(int32_t dtype, const void* A, const void* W, float* C, int32_t M,
                          int32_t N, int32_t K, int32_t tile, void* splitk_scratch,
                          size_t scratch_bytes, alr_stream stream) {
  if (!A || !W || !C || M <= 0 || N <= 0 || K <= 0) return ALR_E_INVALID_ARG;
  if (N % 64 || K % 64) return ALR_E_UNSUPPORTED;
  if (tile < 0 || (tile > 5 && tile < 17) || tile > 20) return ALR_E_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  EpiLogits el;
  el.out = C;
  el.rs = N;
  el.perm = nullptr;
  el.part = nullptr;
  el.part_ld = 0;
  alr_ctx dummy;
  if (dtype == ALR_BF16) {
    const bf16* Wk = (const bf16*)W;
    if (tile == 18 || tile == 20) {  // split-K: partial sums in the scratch buffer
      if (!splitk_scratch || scratch_bytes < (size_t)2 * M * N * 4) return ALR_E_WORKSPACE;
      dummy.splitk_buf = static_cast<float*>(splitk_scratch);
      dummy.splitk_bytes = scratch_bytes;
    }
    launch_gemm<0, bf16>(&dummy, (const bf16*)A, K, Wk, K, M, N, K, el, s, tile);
  } else if (dtype == ALR_F32) {
    launch_gemm<0, float>(&dummy, (const float*)A, K, (const float*)W, K, M, N, K, el, s);
  } else {
    return ALR_E_INVALID_ARG;
  }
  return hipGetLastError() == hipSuccess ? ALR_OK : ALR_E_HIP;
}

static void prof_release(alr_ctx* ctx) {
  for (hipEvent_t e : ctx->prof_ev) (void)hipEventDestroy(e);
  ctx->prof_ev.clear();
  ctx->prof_used = 0;
  ctx->prof_site = 0;
}

alr_status alr_profile_start(alr_ctx* ctx, int32_t site, int32_t capacity) {
  if (!ctx) return ALR_E_INVALID_ARG;
  if (site <= 0 || site >= ALR_PROF_COUNT || capacity <= 0)
    return fail(ctx, ALR_E_INVALID_ARG, "profile site %d / capacity %d invalid", site, capacity);
  prof_release(ctx);
  ctx->prof_ev.resize((size_t)2 * capacity);
  for (auto& e : ctx->prof_ev) {
    const hipError_t err = hipEventCreate(&e);
    if (err != hipSuccess) {
      e = nullptr;
      prof_release(ctx);
      return fail(ctx, ALR_E_HIP, "hipEventCreate failed: %s", hipGetErrorString(err));
    }
  }
  ctx->prof_site = site;
  return ALR_OK;
}

alr_status alr_profile_stop(alr_ctx* ctx, double* total_ms, int32_t* launches) {
  if (!ctx || !total_ms || !launches) return ALR_E_INVALID_ARG;
  double tot = 0.0;
  const size_t n = ctx->prof_used;
  if (n > 0) {
    const hipError_t err = hipEventSynchronize(ctx->prof_ev[2 * n - 1]);
    if (err != hipSuccess) {
      prof_release(ctx);
      return fail(ctx, ALR_E_HIP, "hipEventSynchronize failed: %s", hipGetErrorString(err));
    }
  }
  for (size_t i = 0; i < n; ++i) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, ctx->prof_ev[2 * i], ctx->prof_ev[2 * i + 1]) == hipSuccess)
      tot += ms;
  }
  *total_ms = tot;
  *launches = (int32_t)n;
  prof_release(ctx);
  return ALR_OK;
}

}  // extern "C"
