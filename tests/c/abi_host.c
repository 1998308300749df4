/* The C ABI from a C99 program: the header compiles as C, the library links,
 * and the host-only calls (workspace and scratch sizes, byte-budget
 * capacities, status strings, config validation) work without a GPU.
 * Prints one line per check; exits non-zero on the first failure. */
#include <stdio.h>
#include <string.h>

#include "qevict.h"

#define CHECK(cond, what)                                     \
  do {                                                        \
    if (!(cond)) {                                            \
      printf("FAIL %s: %s\n", what, qevict_last_error());     \
      return 1;                                               \
    }                                                         \
    printf("ok %s\n", what);                                  \
  } while (0)

int main(void) {
  qevict_config cfg;
  memset(&cfg, 0, sizeof cfg);
  cfg.abi_version = QEVICT_ABI_VERSION;
  cfg.batch = 1;
  cfg.num_layers = 1;
  cfg.num_q_heads = 32;
  cfg.num_kv_heads = 8;
  cfg.head_dim = 128;
  cfg.window_tokens = 32;
  cfg.group_size = 32;
  cfg.quant_bits = 2;
  cfg.sink_tokens = 5;
  cfg.recent_tokens = 32;
  cfg.max_context = 32768 + 128;
  cfg.retier_interval = 8;
  cfg.out_dtype = QEVICT_OUT_F32;

  int32_t kf = -1, kq = -1;
  CHECK(qevict_capacities_for_budget(&cfg, 26843545, 700, &kf, &kq) == QEVICT_OK, "capacities");
  CHECK(kf == 61 && kq == 759, "capacities of the 20% budget at q = 0.70");
  cfg.capacity_full = kf;
  cfg.capacity_quant = kq;

  size_t ws = 0, scratch = 0;
  CHECK(qevict_workspace_size(&cfg, &ws) == QEVICT_OK && ws > 0, "workspace size");
  CHECK(qevict_prefill_scores_scratch_size(&cfg, 32768, 32, &scratch) == QEVICT_OK && scratch > 0,
        "prefill score scratch size");

  qevict_config bad = cfg;
  bad.abi_version = QEVICT_ABI_VERSION + 1;
  CHECK(qevict_workspace_size(&bad, &ws) == QEVICT_ERR_UNSUPPORTED, "abi version mismatch rejected");
  bad = cfg;
  bad.window_tokens = 48;
  CHECK(qevict_workspace_size(&bad, &ws) != QEVICT_OK, "window of 48 rejected");
  CHECK(strcmp(qevict_status_string(QEVICT_ERR_CAPACITY), "capacity exceeded") == 0, "status string");
  CHECK(qevict_cache_destroy(NULL) == QEVICT_OK, "destroy(NULL)");
  return 0;
}
