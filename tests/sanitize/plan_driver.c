/*
 * Host-side exercise of the engine's C ABI for the address and
 * undefined-behaviour sanitizers. It drives a MOA_FLAG_PLAN_ONLY engine (no
 * device work) through admission under KV-pool pressure, chunked prefill,
 * histories, both step entry points, partial collects, the inspection hooks
 * and the documented error returns, checking the bookkeeping invariants it
 * can see from outside. Exit status 0 means every check held; the
 * sanitizers abort the process on the first finding.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "moa.h"

#define CHECK(c)                                                        \
  do {                                                                  \
    if (!(c)) {                                                         \
      fprintf(stderr, "plan_driver: check failed at line %d: %s\n", __LINE__, #c); \
      exit(1);                                                          \
    }                                                                   \
  } while (0)

static uint64_t rng_state = 0x9e3779b97f4a7c15ull;
static uint32_t rnd(uint32_t n) { /* splitmix64, reduced */
  uint64_t z = (rng_state += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  z ^= z >> 31;
  return (uint32_t)(z % n);
}

enum { MAXREQ = 512 };
static int32_t want_G[MAXREQ];
static int seen[MAXREQ];

static size_t blob_bytes(const moa_model_cfg* g, size_t esz) {
  const size_t d = g->d_model, qd = (size_t)g->n_heads * g->head_dim, kd = (size_t)g->n_kv_heads * g->head_dim;
  const size_t qkv = qd + 2 * kd, V = g->vocab, F = g->ffn_dim, L = g->n_layers;
  return (2 * V * d + d + L * (2 * d + qkv * d + d * qd + 3 * F * d)) * esz;
}

static int collect_some(moa_engine* e, int64_t* n_done, int64_t n_sub) {
  static moa_result res[MAXREQ];
  static int32_t toks[MAXREQ * 128];
  int32_t n = 0;
  moa_status st = moa_collect(e, -1, res, 1, &n, toks, MAXREQ * 128);
  if (n > 1) {
    CHECK(st == MOA_EINVAL); /* too small: nothing drained, n reports what is ready */
    int32_t n2 = 0;
    CHECK(moa_collect(e, -1, res, MAXREQ, &n2, toks, 0) == MOA_EINVAL && n2 == n);
    st = moa_collect(e, -1, res, MAXREQ, &n, toks, MAXREQ * 128);
  }
  CHECK(st == MOA_OK);
  int64_t off = 0;
  for (int i = 0; i < n; ++i) {
    const int64_t id = res[i].request_id;
    CHECK(id >= 0 && id < n_sub && !seen[id]);
    seen[id] = 1;
    CHECK(res[i].n_tokens == want_G[id]);
    CHECK(res[i].tok_offset == off);
    for (int j = 0; j < res[i].n_tokens; ++j) CHECK(toks[off + j] == -1);
    off += res[i].n_tokens;
    moa_request_info ri;
    CHECK(moa_debug_request(e, id, &ri) == MOA_OK);
    CHECK(ri.state == 3 && ri.finish_step >= ri.admit_step);
  }
  *n_done += n;
  return n;
}

static void run(int32_t dtype, int32_t flags) {
  moa_engine_cfg cfg;
  memset(&cfg, 0, sizeof cfg);
  moa_model_cfg g = {2, 256, 8, 2, 64, 512, 1024, 10000.0f, 1e-5f};
  cfg.model = g;
  cfg.dtype = dtype;
  cfg.kv_block_size = 16;
  cfg.num_kv_blocks = 40;      /* 640 token slots: admission waits for blocks */
  cfg.max_num_seqs = 6;
  cfg.max_prefill_tokens = 100;
  cfg.max_model_len = 700;     /* longer than the pool: ENOSPC is reachable */
  cfg.max_models = 3;
  cfg.flags = MOA_FLAG_PLAN_ONLY | flags;

  size_t arena = 0;
  moa_engine_cfg bad = cfg;
  bad.kv_block_size = 8;
  CHECK(moa_arena_bytes(&bad, &arena) == MOA_EINVAL);
  moa_engine* e = NULL;
  CHECK(moa_create(&bad, NULL, 0, NULL, &e) == MOA_EINVAL && e == NULL);
  CHECK(moa_arena_bytes(&cfg, &arena) == MOA_OK && arena > 0);
  CHECK(moa_create(&cfg, NULL, 0, NULL, &e) == MOA_OK && e != NULL);

  const size_t nb = blob_bytes(&g, dtype == MOA_BF16 ? 2 : 4);
  unsigned char* blob = (unsigned char*)calloc(nb, 1);
  CHECK(blob != NULL);
  int32_t mid = -1;
  CHECK(moa_load_expert(e, &g, blob, nb - 2, &mid) == MOA_EINVAL);
  moa_model_cfg g2 = g;
  g2.ffn_dim = 768;
  CHECK(moa_load_expert(e, &g2, blob, nb, &mid) == MOA_EINVAL);
  for (int m = 0; m < 3; ++m) {
    CHECK(moa_load_expert(e, &g, blob, nb, &mid) == MOA_OK);
    CHECK(mid == m);
  }
  CHECK(moa_load_expert(e, &g, blob, nb, &mid) == MOA_ENOMEM);
  free(blob);

  int32_t prompt[700];
  for (int i = 0; i < 700; ++i) prompt[i] = (int32_t)rnd(1024);
  int64_t rid = -1;
  CHECK(moa_submit(e, prompt, 0, 0, 4, &rid) == MOA_EINVAL);
  CHECK(moa_submit(e, prompt, 10, 0, 0, &rid) == MOA_EINVAL);
  CHECK(moa_submit(e, prompt, 10, 3, 4, &rid) == MOA_EINVAL);
  CHECK(moa_submit(e, prompt, 690, 0, 20, &rid) == MOA_EINVAL); /* beyond max_model_len */
  CHECK(moa_submit(e, prompt, 660, 0, 10, &rid) == MOA_ENOSPC); /* 42 blocks > pool */
  CHECK(moa_submit_with_history(e, 0, 5, -1, NULL, 4, &rid) == MOA_EINVAL);
  CHECK(moa_submit_with_history(e, 9, 5, 10, NULL, 4, &rid) == MOA_EINVAL);

  int64_t n_sub = 0, n_done = 0;
  int64_t last_step = -1;
  for (int round = 0; round < 4; ++round) {
    const int burst = 20 + (int)rnd(20);
    for (int i = 0; i < burst && n_sub < MAXREQ; ++i) {
      const int32_t model = (int32_t)rnd(3);
      int32_t G = 1 + (int32_t)rnd(120);
      moa_status st;
      if (rnd(5) == 0) {
        const int32_t ctx = (int32_t)rnd(400);
        st = moa_submit_with_history(e, model, (int32_t)rnd(1024), ctx, NULL, G, &rid);
      } else {
        const int32_t P = 1 + (int32_t)rnd(450);
        st = moa_submit(e, prompt, P, model, G, &rid);
      }
      if (st == MOA_ENOMEM) break; /* token or block-list store full: collect first */
      CHECK(st == MOA_OK && rid == n_sub);
      want_G[rid] = G;
      n_sub++;
      if (rnd(4) == 0) { /* capture buffers must be at least G * vocab floats */
        float tiny[4];
        CHECK(moa_debug_capture_logits(e, rid, tiny, 4) == MOA_EINVAL);
      }
    }
    for (int s = 0; s < 150; ++s) {
      moa_step_info info;
      const moa_status st = (s % 3 == 2) ? moa_step_noalloc(e, &info) : moa_step(e, &info);
      CHECK(st == MOA_OK);
      if (info.step < 0) break;
      CHECK(info.step == last_step + 1);
      last_step = info.step;
      CHECK(info.running <= cfg.max_num_seqs && info.free_blocks >= 0 && info.free_blocks <= cfg.num_kv_blocks);
      CHECK(info.prefill_tokens <= cfg.max_prefill_tokens);
      int32_t ns = 0, nm = 0, models[3], sm0[5], sr0[5], sl0[5];
      double cost[3];
      CHECK(moa_debug_step_shares(e, &ns, &nm, models, cost, sm0, sr0, sl0) == MOA_OK);
      CHECK(ns >= 1 && ns <= 4 && nm >= 0 && nm <= 3);
      CHECK(sm0[ns] == nm && sr0[ns] == info.prefill_tokens + info.decode_rows);
      for (int u = 0; u < ns; ++u) CHECK(sm0[u] <= sm0[u + 1] && sr0[u] <= sr0[u + 1]);
      if (s % 7 == 0) collect_some(e, &n_done, n_sub);
    }
    /* inspection hooks on every request so far */
    for (int64_t id = 0; id < n_sub; ++id) {
      moa_request_info ri;
      CHECK(moa_debug_request(e, id, &ri) == MOA_OK);
      int32_t bt[64], nbt = -1;
      const moa_status sb = moa_debug_block_table(e, id, bt, 64, &nbt);
      CHECK(sb == MOA_OK || sb == MOA_ESTATE);
      if (sb == MOA_OK) {
        CHECK(nbt >= 0 && nbt <= cfg.num_kv_blocks);
        for (int k = 0; k < nbt; ++k) CHECK(bt[k] >= 0 && bt[k] < cfg.num_kv_blocks);
      }
      int64_t ch[3 * 16];
      int32_t nch = -1;
      const moa_status sc = moa_debug_chunks(e, id, ch, 16, &nch);
      CHECK(sc == MOA_OK || sc == MOA_EINVAL);
    }
    CHECK(moa_debug_request(e, n_sub, NULL) == MOA_EINVAL);
  }
  /* drain */
  for (;;) {
    moa_step_info info;
    CHECK(moa_step(e, &info) == MOA_OK);
    if (info.step < 0) break;
    CHECK(info.step == last_step + 1);
    last_step = info.step;
  }
  while (collect_some(e, &n_done, n_sub) > 0) {
  }
  CHECK(n_done == n_sub);
  for (int64_t id = 0; id < n_sub; ++id) CHECK(seen[id]);
  memset(seen, 0, sizeof seen);

  int64_t n_rows = 0;
  CHECK(moa_debug_steps(e, NULL, 0, &n_rows) == MOA_OK || n_rows >= 0);
  if (n_rows > 0) {
    int64_t* tr = (int64_t*)malloc((size_t)n_rows * 6 * sizeof(int64_t));
    CHECK(tr != NULL);
    int64_t got = 0;
    CHECK(moa_debug_steps(e, tr, n_rows, &got) == MOA_OK && got == n_rows);
    for (int64_t i = 0; i < got; ++i) CHECK(tr[i * 6] == i && tr[i * 6 + 5] >= 0);
    free(tr);
  }
  moa_destroy(e);
  printf("plan_driver: dtype %d flags %d: %lld requests over %lld steps\n", dtype, flags, (long long)n_sub,
         (long long)(last_step + 1));
}

int main(void) {
  run(MOA_F32, 0);
  run(MOA_BF16, 0);                    /* plans the two-stream shares */
  run(MOA_BF16, MOA_FLAG_ONE_STREAM);
  printf("plan_driver: ok\n");
  return 0;
}
