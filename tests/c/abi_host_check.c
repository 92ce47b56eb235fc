/* A plain C client of include/rwttt.h: planning and the owner table on a
 * host-only context (no workspace, so nothing touches a device).  Built and
 * run by tests/test_host_abi.py; prints "ok" and exits 0 on success. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "rwttt.h"

#define CHECK(cond)                                                \
  do {                                                             \
    if (!(cond)) {                                                 \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      return 1;                                                    \
    }                                                              \
  } while (0)

int main(void) {
  enum { OWNERS = 4, LAYERS = 2 };
  const void* w0[LAYERS] = {(const void*)0x10000, (const void*)0x20000};
  void* slots[OWNERS * LAYERS * 2];
  for (int i = 0; i < OWNERS * LAYERS * 2; ++i) slots[i] = (void*)(uintptr_t)(0x1000000 + 0x1000 * i);
  rwttt_config cfg;
  memset(&cfg, 0, sizeof(cfg));
  cfg.n_owners = OWNERS;
  cfg.n_layers = LAYERS;
  cfg.d_ff = 64;
  cfg.d_model = 32;
  cfg.io_dtype = RWTTT_BF16;
  cfg.state_dtype = RWTTT_F32;
  cfg.max_group = 4;
  cfg.backend = RWTTT_FAST_WEIGHT;
  cfg.w0 = w0;
  cfg.slots = slots;
  rwttt_ctx* ctx = NULL;
  CHECK(rwttt_create(&cfg, &ctx) == RWTTT_OK && ctx != NULL);

  /* three READ events and one WRITE event at step 5: one group per effect */
  rwttt_event ev[4];
  memset(ev, 0, sizeof(ev));
  for (uint32_t i = 0; i < 4; ++i) {
    ev[i].owner = 3 - i;
    ev[i].effect = i == 1 ? RWTTT_WRITE : RWTTT_READ;
    ev[i].shape_class = i == 1 ? 7u : 0u;
    ev[i].ready_step = 5;
  }
  rwttt_group groups[4];
  uint32_t omap[4], deferred[4], ng = 0, nm = 0, nd = 0;
  int32_t evst[4];
  CHECK(rwttt_plan(ctx, ev, 4, 5, 0, 0, groups, 4, &ng, omap, 4, &nm, deferred, 4, &nd, evst) == RWTTT_OK);
  CHECK(ng == 2 && nm == 4 && nd == 0);
  CHECK(groups[0].effect == RWTTT_READ && groups[0].count == 3);
  CHECK(omap[0] == 0 && omap[1] == 1 && omap[2] == 3);   /* (ready_step, owner) order */
  CHECK(groups[1].effect == RWTTT_WRITE && omap[3] == 2);

  /* an injected failure opens owner 2's candidate without a launch; it can
     only roll back, which restores its version and live slot */
  void* live = NULL;
  CHECK(rwttt_slot(ctx, 2, 0, 0, &live) == RWTTT_OK);
  CHECK(rwttt_inject_write_failures(ctx, 1) == RWTTT_OK);
  const void* z[1] = {(const void*)0x100};
  const void* g[1] = {(const void*)0x200};
  /* a member planned at a version other than V(r) is refused before anything changes */
  const uint64_t stale[4] = {0, 0, 0, 1};
  CHECK(rwttt_write(ctx, &groups[1], omap, stale, 0, 4, z, g, 1.0f, NULL, NULL, NULL) == RWTTT_E_STALE_VERSION);
  const uint64_t planned[4] = {0, 0, 0, 0};
  CHECK(rwttt_write(ctx, &groups[1], omap, planned, 0, 4, z, g, 1.0f, NULL, NULL, NULL) == RWTTT_E_WRITE_FAILED);
  uint64_t v = 99;
  int32_t dirty = 0;
  CHECK(rwttt_version(ctx, 2, &v, &dirty) == RWTTT_OK && v == 0 && dirty == 1);
  CHECK(rwttt_commit(ctx, omap + 3, 1) == RWTTT_E_WRITE_FAILED);
  CHECK(rwttt_rollback(ctx, omap + 3, 1) == RWTTT_OK);
  void* live2 = NULL;
  CHECK(rwttt_slot(ctx, 2, 0, 0, &live2) == RWTTT_OK && live2 == live);
  CHECK(rwttt_version(ctx, 2, &v, &dirty) == RWTTT_OK && v == 0 && dirty == 0);

  /* a host-only context refuses device work */
  CHECK(rwttt_read(ctx, &groups[0], omap, NULL, 0, (const void*)0x1000, (void*)0x2000, NULL) == RWTTT_E_INVALID);
  CHECK(rwttt_read(ctx, &groups[0], omap, stale, 0, (const void*)0x1000, (void*)0x2000, NULL) == RWTTT_E_INVALID);
  const uint64_t stale_read[4] = {0, 5, 0, 0};
  CHECK(rwttt_read(ctx, &groups[0], omap, stale_read, 0, (const void*)0x1000, (void*)0x2000, NULL) ==
        RWTTT_E_STALE_VERSION);
  CHECK(rwttt_fork(ctx, 0, 1, NULL) == RWTTT_E_INVALID);
  CHECK(strlen(rwttt_strerror(RWTTT_E_STALE_VERSION)) > 0);

  size_t ws = 0, sb = 0;
  CHECK(rwttt_workspace_bytes(&cfg, &ws) == RWTTT_OK && ws > 0);
  CHECK(rwttt_slot_bytes(&cfg, &sb) == RWTTT_OK && sb == 64u * 32u * 4u);
  cfg.backend = RWTTT_DELTA_ADAPTER;
  cfg.rank = 8;
  CHECK(rwttt_slot_bytes(&cfg, &sb) == RWTTT_OK && sb == (64u + 32u) * 8u * 4u);
  cfg.rank = RWTTT_MAX_RANK + 1;
  CHECK(rwttt_slot_bytes(&cfg, &sb) == RWTTT_E_INVALID);

  CHECK(rwttt_destroy(ctx) == RWTTT_OK);
  printf("ok\n");
  return 0;
}
