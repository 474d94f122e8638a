/* A C11 caller of the library's host-only entry points: the header compiles
 * as C, the symbols link, and parameter validation answers without a GPU.
 * Built and run by tests/test_abi.py::test_header_compiles_and_links_as_c. */
#include <stdio.h>
#include <string.h>

#include "snapstream.h"

int main(void) {
  snap_params p;
  memset(&p, 0, sizeof(p));
  p.n_q_heads = 32;
  p.n_kv_heads = 8;
  p.d_qk = 128;
  p.d_v = 128;
  p.sink = 4;
  p.recent = 1024;
  p.topk = 2048;
  p.obs_window = 32;
  p.pool_kernel = 7;
  p.pool = SNAP_POOL_MAX;
  p.norm = SNAP_NORM_CAND;
  p.in_dtype = SNAP_BF16;
  p.kv_dtype = SNAP_BF16;
  p.kv_reuse = SNAP_KV_AUTO;
  const size_t wc = snap_compress_workspace(&p, 2, 4096);
  const size_t wd = snap_decode_workspace(&p, 2);
  printf("compress_ws %zu decode_ws %zu\n", wc, wd);
  /* an even pool kernel is refused before anything touches a device */
  p.pool_kernel = 4;
  snap_cache c;
  memset(&c, 0, sizeof(c));
  const snap_status st = snap_decode_attn(&p, &c, NULL, NULL, 1, NULL, NULL, NULL, SNAP_BF16, NULL, 0, NULL);
  printf("status %d %s | %s\n", (int)st, snap_status_str(st), snap_last_error());
  return (wc > 0 && wd > 0 && st == SNAP_ERR_INVALID_ARG) ? 0 : 1;
}
