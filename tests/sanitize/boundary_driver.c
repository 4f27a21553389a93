/* Drives the C-ABI's host-side argument checks (no kernel launches: every
 * call here is rejected before one), for a build of the library whose host
 * code carries AddressSanitizer and UndefinedBehaviorSanitizer. Exits non-zero
 * if a call returns another status than the one its arguments call for. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "dcp.h"

static int failures = 0;
static void expect(int got, int want, const char* what) {
  if (got != want) {
    fprintf(stderr, "FAILED: %s: status %d, expected %d (%s)\n", what, got, want, dcp_last_error());
    ++failures;
  } else if (want != DCP_OK && strlen(dcp_last_error()) == 0) {
    fprintf(stderr, "FAILED: %s: no error message\n", what);
    ++failures;
  }
}

int main(void) {
  size_t bytes = 0;
  float fake_f[16];
  int32_t fake_i[16];
  dcp_shape sh = {24000, 384, 128, 16, 24, DCP_BF16, DCP_F32, 1e-5f};
  dcp_weights w = {fake_f, fake_f, fake_f, fake_f, fake_f, NULL, NULL, NULL};
  expect(strlen(dcp_version()) > 0 ? DCP_OK : -99, DCP_OK, "version");
  expect(dcp_workspace_size(&sh, 24000, 6, &bytes), DCP_OK, "workspace size");
  expect(bytes > 0 ? DCP_OK : -99, DCP_OK, "workspace size > 0");
  expect(dcp_workspace_size(&sh, 24000, 6, NULL), DCP_ERR_INVALID_ARGUMENT, "workspace size, null out");
  expect(dcp_workspace_size(NULL, 24000, 6, &bytes), DCP_ERR_INVALID_ARGUMENT, "workspace size, null shape");
  expect(dcp_workspace_size(&sh, 24000, 0, &bytes), DCP_ERR_INVALID_ARGUMENT, "zero key blocks");
  dcp_shape bad = sh;
  bad.c_z = 0;
  expect(dcp_workspace_size(&bad, 10, 1, &bytes), DCP_ERR_INVALID_ARGUMENT, "c_z = 0");
  bad = sh;
  bad.ln_eps = -1.0f;
  expect(dcp_workspace_size(&bad, 10, 1, &bytes), DCP_ERR_INVALID_ARGUMENT, "negative eps");
  expect(dcp_pair_bias_attention(NULL, &w, fake_f, fake_f, NULL, 0, 10, 1, fake_f, fake_f, 1 << 20, NULL),
         DCP_ERR_INVALID_ARGUMENT, "attention, null shape");
  expect(dcp_pair_bias_attention(&sh, &w, fake_f, fake_f, NULL, 23990, 20, 1, fake_f, fake_f, 1 << 20, NULL),
         DCP_ERR_INVALID_ARGUMENT, "attention, rows past N");
  expect(dcp_pair_bias_attention(&sh, NULL, fake_f, fake_f, NULL, 0, 10, 1, fake_f, fake_f, 1 << 20, NULL),
         DCP_ERR_INVALID_ARGUMENT, "attention, null weights");
  dcp_sparse_shape ss = {96000, 128, 16, 4, 32, 128, DCP_BF16, DCP_F32, 0, 1e-5f};
  expect(dcp_sparse_workspace_size(&ss, 24000, &bytes), DCP_OK, "sparse workspace size");
  ss.k = 0;
  expect(dcp_sparse_workspace_size(&ss, 24000, &bytes), DCP_ERR_INVALID_ARGUMENT, "sparse k = 0");
  expect(dcp_knn_topk(NULL, 10, fake_f, 10, 0, -1, NULL, NULL, 0, 4, fake_i, fake_f, NULL, 0, NULL), DCP_ERR_INVALID_ARGUMENT,
         "knn, null queries");
  expect(dcp_knn_topk(fake_f, 10, fake_f, 10, 0, -1, NULL, NULL, 0, 0, fake_i, fake_f, NULL, 0, NULL),
         DCP_ERR_INVALID_ARGUMENT, "knn, k = 0");
  expect(dcp_knn_topk(fake_f, 10, fake_f, 10, 0, -1, NULL, NULL, 1, 4, fake_i, fake_f, NULL, 0, NULL),
         DCP_ERR_INVALID_ARGUMENT, "knn, group mode without groups");
  expect(dcp_knn_topk(fake_f, 10, fake_f, 10, 0, -1, NULL, NULL, 0, 4, fake_i, fake_f, NULL, 0, NULL),
         DCP_ERR_WORKSPACE, "knn, no workspace");
  expect(dcp_knn_workspace_size(96000, &bytes), DCP_OK, "knn workspace size");
  expect(bytes == 96000 * 16 + 750 * 32 ? DCP_OK : -99, DCP_OK, "knn workspace size value");
  expect(dcp_knn_workspace_size(-1, &bytes), DCP_ERR_INVALID_ARGUMENT, "knn workspace size, n_c < 0");
  expect(dcp_topk_merge(4, 0, fake_i, fake_f, fake_i, fake_f, fake_i, fake_f, NULL), DCP_ERR_INVALID_ARGUMENT,
         "topk merge, k = 0");
  expect(dcp_transition_workspace_size(128, 512, DCP_BF16, &bytes), DCP_OK, "transition workspace size");
  expect(dcp_transition_workspace_size(96, 512, DCP_BF16, &bytes), DCP_ERR_UNSUPPORTED, "transition bf16 c_z 96");
  expect(dcp_pair_transition(10, 128, 512, DCP_BF16, 1e-5f, NULL, fake_f, fake_f, NULL, NULL, fake_f, fake_f, fake_f,
                             1 << 20, NULL),
         DCP_ERR_INVALID_ARGUMENT, "transition, null w1");
  expect(dcp_scatter_mean_workspace_size(24000, 128, &bytes), DCP_OK, "pooling workspace size");
  expect(dcp_scatter_mean_workspace_size(24000, 0, &bytes), DCP_ERR_INVALID_ARGUMENT, "pooling c = 0");
  expect(dcp_scatter_mean(10, 4, 600, DCP_F32, DCP_F32, fake_f, fake_i, fake_f, fake_f, 1 << 20, NULL),
         DCP_ERR_UNSUPPORTED, "pooling c = 600");
  expect(dcp_set_timing_events(NULL, NULL), DCP_OK, "timing events cleared");
  if (failures) return 1;
  printf("boundary driver: all checks behaved\n");
  return 0;
}
