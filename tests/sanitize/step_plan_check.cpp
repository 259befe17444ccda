// Host-side check of the per-step work lists the engine hands to its
// attention, combine and LM-head kernels. It includes the engine's source
// (the lists are internal to it), drives MOA_FLAG_PLAN_ONLY engines through
// random schedules (prompts, chunked prefill, injected histories up to 33k
// positions, KV-pool pressure, one to four model streams, both dtypes) and,
// after every step, checks against the request bookkeeping:
//   * rows: grouped by model in one contiguous run per model, each row's
//     position, block list and model those of its request, and the token it
//     reads already written (a prompt token, or an output emitted in an
//     earlier step);
//   * decode attention: every row's keys [0, pos] covered exactly once by its
//     items, each decode range within one 256-key split (an f32 engine's
//     prompt rows take one item over all their keys) and starting on a KV block
//     boundary whose block-list offset is the row's list plus k0 / 16, inside
//     the request's blocks; one final writer per row (an unsplit item, or a
//     combine item over exactly the row's partial slots); partial slots
//     unique and below the workspace's slot capacity;
//   * causal prefill blocks (bf16): every prompt row in exactly one block of
//     at most 128 consecutive positions of one request;
//   * LM rows: each decode row and each prompt's last row once, writing the
//     request's next output slot;
//   * launch order and model-stream shares: items by share, then by
//     decreasing key-range length; combine items by decreasing slot count;
//     share boundaries on model-group boundaries; every list within the
//     capacities the workspace was sized for.
// No HIP call is made.
#include "../../paper_2606_03014_amd/csrc/engine.cpp"

#include <cstdlib>
#include <map>
#include <set>

namespace {

uint64_t g_rng = 0x452821e638d01377ull;
uint32_t rnd(uint32_t n) {  // splitmix64, reduced
  uint64_t z = (g_rng += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  z ^= z >> 31;
  return (uint32_t)(z % n);
}

#define CHECK(c, ...)                                                         \
  do {                                                                        \
    if (!(c)) {                                                               \
      std::fprintf(stderr, "step_plan_check: line %d: %s: ", __LINE__, #c);   \
      std::fprintf(stderr, __VA_ARGS__);                                      \
      std::fprintf(stderr, "\n");                                             \
      std::exit(1);                                                           \
    }                                                                         \
  } while (0)

size_t blob_bytes(const moa_model_cfg& g, size_t esz) {
  const size_t d = g.d_model, qd = (size_t)g.n_heads * g.head_dim, kd = (size_t)g.n_kv_heads * g.head_dim;
  const size_t qkv = qd + 2 * kd, V = g.vocab, F = g.ffn_dim, L = g.n_layers;
  return (2 * V * d + d + L * (2 * d + qkv * d + d * qd + 3 * F * d)) * esz;
}

struct Tracker {
  std::vector<int64_t> produced;   // outputs emitted so far, per request
};

void check_step(const moa_engine* e, int64_t s, Tracker& tr) {
  const int T = (int)e->r_tok.size();
  const int R = (int)e->l_src.size();
  CHECK(T <= e->lay.Tmax && R <= e->lay.Rmax, "step %lld: %d rows, %d LM rows", (long long)s, T, R);
  CHECK((int64_t)e->items.size() <= e->lay.items_cap, "step %lld: %zu items", (long long)s, e->items.size());
  // live requests of this step by block-list offset (unique while they live)
  std::map<int64_t, const Request*> by_bt;
  for (const Request& r : e->reqs)
    if (r.state == 1 || (r.state == 2 && r.finish_step == s)) {
      CHECK(by_bt.emplace(r.bt_off, &r).second, "step %lld: two live requests at block list %lld", (long long)s,
            (long long)r.bt_off);
    }
  auto req_of = [&](int row) {
    auto it = by_bt.find(e->r_bt[row]);
    CHECK(it != by_bt.end(), "step %lld: row %d names block list %d of no live request", (long long)s, row,
          e->r_bt[row]);
    return it->second;
  };
  // rows
  std::set<int> seen_models;
  std::vector<int> row_kind(T);   // 0 prefill, 1 decode
  for (int row = 0; row < T; ++row) {
    const Request* r = req_of(row);
    const int m = e->r_model[row];
    if (row == 0 || e->r_model[row - 1] != m) {
      CHECK(seen_models.insert(m).second, "step %lld: model %d rows not contiguous", (long long)s, m);
    }
    CHECK(r->model == m, "step %lld: row %d model %d, request model %d", (long long)s, row, m, r->model);
    const int pos = e->r_pos[row];
    CHECK(pos >= 0 && pos < r->P + r->G - 1, "step %lld: row %d position %d (P %d G %d)", (long long)s, row, pos,
          r->P, r->G);
    row_kind[row] = (r->history || pos >= r->P) ? 1 : 0;   // a history's seed row decodes
    const int64_t idx = e->r_tok[row] - r->tok_off;
    const int prompt_slots = r->P - r->shift;
    CHECK(idx == pos - r->shift, "step %lld: row %d reads slot %lld for position %d", (long long)s, row,
          (long long)idx, pos);
    if (idx >= prompt_slots)
      CHECK(idx - prompt_slots < tr.produced[r->id], "step %lld: row %d reads output %lld, %lld produced",
            (long long)s, row, (long long)(idx - prompt_slots), (long long)tr.produced[r->id]);
    CHECK((pos + kBlock) / kBlock <= r->need, "step %lld: row %d position %d beyond %d blocks", (long long)s, row,
          pos, r->need);
  }
  // decode attention items and the split combine
  const bool tiled = e->bf16 && (e->cfg.model.head_dim == 64 || e->cfg.model.head_dim == 128);
  std::vector<std::vector<std::pair<int, int>>> ranges(T);
  std::vector<int> finals(T, 0);
  std::map<int, int> slot_row;
  for (const AttnItem& it : e->items) {
    CHECK(it.row >= 0 && it.row < T, "step %lld: item row %d", (long long)s, it.row);
    const int ctx = e->r_pos[it.row] + 1;
    CHECK(!(tiled && row_kind[it.row] == 0), "step %lld: prompt row %d has a decode item", (long long)s, it.row);
    CHECK(it.k0 >= 0 && it.k0 < it.k1 && it.k1 <= ctx && it.k0 % kBlock == 0, "step %lld: row %d keys [%d, %d) of %d",
          (long long)s, it.row, it.k0, it.k1, ctx);
    // decode rows read their keys in 256-key splits; f32 prompt rows whole
    if (it.slot >= 0 || row_kind[it.row] == 1)
      CHECK(it.k0 / kSplitKeys == (it.k1 - 1) / kSplitKeys, "step %lld: row %d keys [%d, %d) cross a split",
            (long long)s, it.row, it.k0, it.k1);
    CHECK(it.bt_off == e->r_bt[it.row] + it.k0 / kBlock, "step %lld: row %d item block offset %d", (long long)s,
          it.row, it.bt_off);
    ranges[it.row].push_back({it.k0, it.k1});
    if (it.slot < 0) {
      CHECK(it.k0 == 0 && it.k1 == ctx, "step %lld: row %d writes its output from keys [%d, %d)", (long long)s,
            it.row, it.k0, it.k1);
      finals[it.row]++;
    } else {
      CHECK(it.slot < e->lay.slots_cap, "step %lld: slot %d of %lld", (long long)s, it.slot,
            (long long)e->lay.slots_cap);
      CHECK(slot_row.emplace(it.slot, it.row).second, "step %lld: slot %d written twice", (long long)s, it.slot);
    }
  }
  for (const ReduceItem& rd : e->red) {
    CHECK(rd.row >= 0 && rd.row < T && rd.nslots >= 2, "step %lld: combine row %d over %d slots", (long long)s,
          rd.row, rd.nslots);
    const int ctx = e->r_pos[rd.row] + 1;
    CHECK(rd.nslots == (ctx + kSplitKeys - 1) / kSplitKeys, "step %lld: row %d: %d slots for %d keys", (long long)s,
          rd.row, rd.nslots, ctx);
    for (int k = 0; k < rd.nslots; ++k) {
      auto it = slot_row.find(rd.slot0 + k);
      CHECK(it != slot_row.end() && it->second == rd.row, "step %lld: row %d combines slot %d not its own",
            (long long)s, rd.row, rd.slot0 + k);
      slot_row.erase(it);
    }
    finals[rd.row]++;
  }
  CHECK(slot_row.empty(), "step %lld: %zu partial slots never combined", (long long)s, slot_row.size());
  for (int row = 0; row < T; ++row) {
    const int ctx = e->r_pos[row] + 1;
    if (tiled && row_kind[row] == 0) {
      CHECK(ranges[row].empty() && finals[row] == 0, "step %lld: prompt row %d in decode lists", (long long)s, row);
      continue;
    }
    CHECK(finals[row] == 1, "step %lld: row %d has %d final writers", (long long)s, row, finals[row]);
    std::sort(ranges[row].begin(), ranges[row].end());
    int end = 0;
    for (auto& rg : ranges[row]) {
      CHECK(rg.first == end, "step %lld: row %d keys jump to %d at %d", (long long)s, row, rg.first, end);
      end = rg.second;
    }
    CHECK(end == ctx, "step %lld: row %d keys end at %d of %d", (long long)s, row, end, ctx);
  }
  // causal prefill blocks
  std::vector<int> in_block(T, 0);
  for (const PrefillItem& pi : e->pitems) {
    CHECK(tiled, "step %lld: prefill blocks in an untiled engine", (long long)s);
    CHECK(pi.nq >= 1 && pi.nq <= kPrefillRows && pi.row0 >= 0 && pi.row0 + pi.nq <= T,
          "step %lld: prefill block rows [%d, +%d)", (long long)s, pi.row0, pi.nq);
    for (int i = 0; i < pi.nq; ++i) {
      const int row = pi.row0 + i;
      CHECK(e->r_bt[row] == pi.bt_off && e->r_pos[row] == pi.pos0 + i && row_kind[row] == 0,
            "step %lld: prefill block at row %d: row %d is not position %d of its request", (long long)s, pi.row0,
            row, pi.pos0 + i);
      in_block[row]++;
    }
  }
  if (tiled)
    for (int row = 0; row < T; ++row)
      CHECK(in_block[row] == (row_kind[row] == 0 ? 1 : 0), "step %lld: row %d in %d prefill blocks", (long long)s,
            row, in_block[row]);
  // LM rows
  std::set<int> lm_rows;
  std::map<int64_t, int64_t> emitted;
  for (int i = 0; i < R; ++i) {
    const int row = e->l_src[i];
    CHECK(row >= 0 && row < T && lm_rows.insert(row).second, "step %lld: LM row %d", (long long)s, row);
    const Request* r = req_of(row);
    CHECK(row_kind[row] == 1 || e->r_pos[row] == r->P - 1, "step %lld: LM row %d at position %d of %d",
          (long long)s, row, e->r_pos[row], r->P);
    const int64_t out = e->l_dst[i] - r->tok_off - (r->P - r->shift);
    CHECK(out == tr.produced[r->id] + emitted[r->id] && out < r->G, "step %lld: request %lld writes output %lld",
          (long long)s, (long long)r->id, (long long)out);
    emitted[r->id]++;
  }
  for (int row = 0; row < T; ++row)
    if (row_kind[row] == 1) CHECK(lm_rows.count(row), "step %lld: decode row %d emits nothing", (long long)s, row);
  for (auto& kv : emitted) {
    CHECK(kv.second == 1, "step %lld: request %lld emits %lld tokens", (long long)s, (long long)kv.first,
          (long long)kv.second);
    tr.produced[kv.first] += kv.second;
  }
  // launch order and shares
  const int ns = e->nshare;
  CHECK(ns >= 1 && ns <= kMaxShares && e->sh_row[0] == 0 && e->sh_row[ns] == T && e->sh_lm[ns] == R,
        "step %lld: %d shares", (long long)s, ns);
  for (int u = 0; u < ns; ++u) {
    CHECK(e->sh_row[u] <= e->sh_row[u + 1], "step %lld: share rows", (long long)s);
    const int b = e->sh_row[u];
    if (b > 0 && b < T)
      CHECK(e->r_model[b] != e->r_model[b - 1], "step %lld: share %d starts inside model %d's rows", (long long)s, u,
            e->r_model[b]);
    for (int i = e->sh_item[u]; i < e->sh_item[u + 1]; ++i) {
      const AttnItem& it = e->items[i];
      CHECK(it.row >= e->sh_row[u] && it.row < e->sh_row[u + 1], "step %lld: item %d outside share %d", (long long)s,
            i, u);
      if (i > e->sh_item[u])
        CHECK(it.k1 - it.k0 <= e->items[i - 1].k1 - e->items[i - 1].k0, "step %lld: item %d longer than the last",
              (long long)s, i);
    }
    for (int i = e->sh_red[u]; i < e->sh_red[u + 1]; ++i) {
      CHECK(e->red[i].row >= e->sh_row[u] && e->red[i].row < e->sh_row[u + 1], "step %lld: combine %d outside share",
            (long long)s, i);
      if (i > e->sh_red[u]) CHECK(e->red[i].nslots <= e->red[i - 1].nslots, "step %lld: combine order", (long long)s);
    }
    for (int i = e->sh_pre[u]; i < e->sh_pre[u + 1]; ++i)
      CHECK(e->pitems[i].row0 >= e->sh_row[u] && e->pitems[i].row0 < e->sh_row[u + 1],
            "step %lld: prefill block %d outside share", (long long)s, i);
    for (int i = e->sh_lm[u]; i < e->sh_lm[u + 1]; ++i)
      CHECK(e->l_src[i] >= e->sh_row[u] && e->l_src[i] < e->sh_row[u + 1], "step %lld: LM row %d outside share",
            (long long)s, i);
  }
  CHECK(e->sh_item[ns] == (int)e->items.size() && e->sh_red[ns] == (int)e->red.size() &&
            e->sh_pre[ns] == (int)e->pitems.size(),
        "step %lld: share bounds do not end at the lists' ends", (long long)s);
}

void run(int32_t dtype, int32_t hd, int32_t flags, int n_req) {
  moa_engine_cfg cfg{};
  moa_model_cfg g = {2, 256, 256 / hd * 2, 2, hd, 512, 1024, 10000.0f, 1e-5f};
  cfg.model = g;
  cfg.dtype = dtype;
  cfg.kv_block_size = kBlock;
  cfg.num_kv_blocks = 3000 + (int)rnd(6000);     // 48k..144k positions: histories queue for blocks
  cfg.max_num_seqs = 4 + (int)rnd(60);
  cfg.max_prefill_tokens = 64 + (int)rnd(3000);
  cfg.max_model_len = 34000;
  cfg.max_models = 1 + (int)rnd(kMaxModels);
  cfg.flags = MOA_FLAG_PLAN_ONLY | flags;
  moa_engine* e = nullptr;
  CHECK(moa_create(&cfg, nullptr, 0, nullptr, &e) == MOA_OK, "create");
  const size_t nb = blob_bytes(g, dtype == MOA_BF16 ? 2 : 4);
  std::vector<unsigned char> blob(nb, 0);
  for (int m = 0; m < cfg.max_models; ++m) {
    int32_t mid = -1;
    CHECK(moa_load_expert(e, &g, blob.data(), nb, &mid) == MOA_OK && mid == m, "load %d", m);
  }
  std::vector<int32_t> prompt(6000);
  for (auto& t : prompt) t = (int32_t)rnd(1024);
  Tracker tr;
  int64_t steps = 0, rows = 0, items = 0, submitted = 0, multi_share = 0, split_rows = 0, max_keys = 0;
  int64_t last = -1;
  std::vector<moa_result> res(4096);
  std::vector<int32_t> toks(1 << 20);
  while (submitted < n_req || !e->pending.empty() || !e->running.empty()) {
    // arrivals
    const int burst = submitted < n_req ? (int)rnd(6) : 0;
    for (int i = 0; i < burst && submitted < n_req; ++i) {
      const int32_t model = (int32_t)rnd((uint32_t)cfg.max_models);
      const int32_t G = 1 + (int32_t)rnd(rnd(4) == 0 ? 600 : 40);
      int64_t rid = -1;
      moa_status st;
      if (rnd(3) == 0) {
        const int32_t ctx = rnd(2) ? (int32_t)rnd(2000) : 20000 + (int32_t)rnd(13000);
        st = moa_submit_with_history(e, model, (int32_t)rnd(1024), ctx, nullptr, G, &rid);
      } else {
        const int32_t P = 1 + (int32_t)rnd(rnd(3) == 0 ? 5999 : 300);
        st = moa_submit(e, prompt.data(), P, model, G, &rid);
      }
      if (st == MOA_ENOSPC) continue;        // larger than the whole pool
      if (st == MOA_ENOMEM) break;           // stores full: collect first
      CHECK(st == MOA_OK, "submit %d", (int)st);
      if ((int64_t)tr.produced.size() <= rid) tr.produced.resize(rid + 1, 0);
      ++submitted;
    }
    moa_step_info info;
    const moa_status st = (steps % 3 == 2) ? moa_step_noalloc(e, &info) : moa_step(e, &info);
    CHECK(st == MOA_OK, "step %d", (int)st);
    if (info.step < 0) {
      if (submitted >= n_req) break;
      continue;
    }
    CHECK(info.step == last + 1, "step order");
    last = info.step;
    check_step(e, info.step, tr);
    ++steps;
    rows += (int64_t)e->r_tok.size();
    items += (int64_t)e->items.size() + (int64_t)e->pitems.size();
    multi_share += e->nshare > 1;
    split_rows += (int64_t)e->red.size();
    for (int p : e->r_pos) max_keys = std::max<int64_t>(max_keys, p + 1);
    if (steps % 5 == 0) {
      int32_t n = 0;
      CHECK(moa_collect(e, -1, res.data(), (int32_t)res.size(), &n, toks.data(), (int64_t)toks.size()) == MOA_OK,
            "collect");
      for (int i = 0; i < n; ++i)
        CHECK(tr.produced[res[i].request_id] == res[i].n_tokens, "request %lld: %lld produced, %d collected",
              (long long)res[i].request_id, (long long)tr.produced[res[i].request_id], res[i].n_tokens);
    }
  }
  moa_destroy(e);
  // the schedule reached what it is meant to exercise
  CHECK(split_rows > 0 && max_keys > 20000, "no long-context split rows");
  // (several model streams: bf16 engines holding two or more models)
  const bool streams = dtype == MOA_BF16 && !(flags & MOA_FLAG_ONE_STREAM) && cfg.max_models > 1;
  CHECK(streams ? multi_share > 0 : multi_share == 0, "%lld steps on several model streams", (long long)multi_share);
  std::printf("step_plan_check: dtype %d head_dim %d flags %d: %lld requests, %lld steps, %lld rows, %lld items, "
              "%lld split rows, %lld multi-stream steps, up to %lld keys\n",
              dtype, hd, flags, (long long)submitted, (long long)steps, (long long)rows, (long long)items,
              (long long)split_rows, (long long)multi_share, (long long)max_keys);
}

}  // namespace

int main(int argc, char** argv) {
  const int n_req = argc > 1 ? std::atoi(argv[1]) : 300;
  if (argc > 2) g_rng ^= std::strtoull(argv[2], nullptr, 10) * 0x9e3779b97f4a7c15ull;   // another seed
  run(MOA_F32, 64, 0, n_req);
  run(MOA_BF16, 64, 0, n_req);
  run(MOA_BF16, 128, 0, n_req);
  run(MOA_BF16, 128, MOA_FLAG_ONE_STREAM, n_req);
  std::printf("step_plan_check: ok\n");
  return 0;
}
