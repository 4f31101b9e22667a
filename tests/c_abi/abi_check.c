/* The C ABI from a plain C99 program: include/alr.h and alr_debug.h compile as
 * C, libalr.so links, and the host-only entry points (validation, sizing,
 * status strings, the decode work plan) answer without a GPU.  Exit code 0 on
 * success; a message and a non-zero code on the first failed check. */
#include <stdio.h>
#include <string.h>

#include "alr.h"
#include "alr_debug.h"

#define CHECK(cond, ...)                  \
  do {                                    \
    if (!(cond)) {                        \
      printf("FAILED: " __VA_ARGS__);     \
      printf("\n");                       \
      return 1;                           \
    }                                     \
  } while (0)

int main(void) {
  alr_config c;
  memset(&c, 0, sizeof c);
  c.n_layers = 2;
  c.d_model = 256;
  c.n_heads = 8;
  c.n_kv_heads = 2;
  c.head_dim = 128;
  c.d_ffn = 512;
  c.vocab = 2048;
  c.rms_eps = 1e-6f;
  c.rope_base = 10000.f;
  c.dtype = ALR_BF16;
  c.max_pos = 4096;
  c.n_feat = 2;
  c.feat_layers[0] = 0;
  c.feat_layers[1] = 1;
  char msg[256];
  CHECK(alr_check_config(&c, msg, sizeof msg) == ALR_OK, "valid config rejected: %s", msg);

  const alr_limits lim = {600, 2, 12, 5};
  const size_t ws = alr_workspace_bytes(&c, &lim);
  CHECK(ws > 0, "workspace bytes 0 for a valid config");
  const alr_limits lim2 = {1200, 2, 12, 5};
  CHECK(alr_workspace_bytes(&c, &lim2) > ws, "workspace does not grow with max_tokens");

  alr_config bad = c;
  bad.n_heads = 7; /* not a multiple of n_kv_heads */
  CHECK(alr_check_config(&bad, msg, sizeof msg) == ALR_E_INVALID_ARG, "7/2 heads accepted");
  CHECK(alr_workspace_bytes(&bad, &lim) == 0, "workspace bytes for an invalid config");

  const int32_t seq_len[2] = {300, 300};
  const int32_t a_seq[3] = {0, 1, 1};
  const int32_t a_pos[3] = {0, 299, 150};
  CHECK(alr_check_rollout(&c, &lim, 2, seq_len, 3, a_seq, a_pos, 5, msg, sizeof msg) == ALR_OK,
        "valid rollout rejected: %s", msg);
  const int32_t a_far[3] = {0, 300, 150}; /* position 300 of a 300-token sequence */
  CHECK(alr_check_rollout(&c, &lim, 2, seq_len, 3, a_seq, a_far, 5, msg, sizeof msg) ==
            ALR_E_OUT_OF_RANGE,
        "anchor past the sequence accepted");

  CHECK(strcmp(alr_status_string(ALR_E_HIP), "ALR_E_HIP") == 0, "status string");
  CHECK(alr_set_rollout_graphs(NULL, 1) == ALR_E_INVALID_ARG, "graph switch on a NULL context");

  int32_t ct = 0, makespan = 0, n_items = 0, items[6 * 256];
  CHECK(alr_debug_decode_plan(&c, 256, 2, seq_len, 3, a_seq, a_pos, &ct, &makespan, &n_items,
                              items, 256) == ALR_OK,
        "decode plan");
  CHECK(n_items > 0 && ct > 0, "empty decode plan");
  printf("ok: workspace %zu bytes, decode plan %d items of %d tiles\n", ws, n_items, ct);
  return 0;
}
