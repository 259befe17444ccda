// Host-side check of the grouped-GEMM planner against the launch contract of
// the GEMM kernels. It includes the engine's source (the planner is internal
// to it) and, for random ragged row mixes on the 8B, 1B and a small model's
// projection shapes in both engine dtypes, plans every projection of a step,
// whole and split into contiguous model-stream shares, then checks:
//   * the tile code is one the GEMM launcher dispatches, with the divisibility
//     and k-split bounds it enforces;
//   * replaying each kernel's own item decode (group lookup by first item,
//     then row chunk / column block / k-split) over every item of the grid
//     covers every (row, column block, k-split) of every carried group exactly
//     once, with no item resolving to an empty group or an empty row range;
//   * the k-splits tile the reduction dimension (the workgroup-tile kernel's
//     equal splits of whole 4-step stages, the medium-M kernel's rounded ones);
//   * split-K partials stay inside the engine's partial buffer;
//   * a share's launch picks the same tiling, split and partial stride as the
//     whole step, so its partials land where the step's consumer reads them;
//   * gate-up (SwiGLU epilogue) is never split and, on the medium-M kernel,
//     fits one workgroup per CU;
//   * the large-M k-split still picks the splits measured best on the GPU.
// The decode below restates the kernels' index arithmetic: a change to either
// side that breaks the contract fails here, on the CPU. No HIP call is made.
#include "../../paper_2606_03014_amd/csrc/engine.cpp"

#include <cstdlib>

namespace {

uint64_t g_rng = 0x243f6a8885a308d3ull;
uint32_t rnd(uint32_t n) {  // splitmix64, reduced
  uint64_t z = (g_rng += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  z ^= z >> 31;
  return (uint32_t)(z % n);
}

int g_fail = 0;
#define CHECK(c, ...)                                                          \
  do {                                                                         \
    if (!(c)) {                                                                \
      std::fprintf(stderr, "gemm_plan_check: line %d: %s: ", __LINE__, #c);    \
      std::fprintf(stderr, __VA_ARGS__);                                       \
      std::fprintf(stderr, "\n");                                              \
      if (++g_fail > 20) std::exit(1);                                         \
      return false;                                                            \
    }                                                                          \
  } while (0)

struct Proj { const char* name; int K, N, epi; bool split; bool lm; };

struct Shape { const char* name; moa_model_cfg m; };

// The tile geometry a (mt, nt) code stands for, as the launcher reads it.
struct Tile { int kind; int rows; int cols; int S; };   // kind 0 f32, 1 workgroup-tile, 2 medium-M

bool dispatchable(bool bf16, const GemmArgs& a, int epi, int mt, int nt, Tile& t, const char* what) {
  const int KS = a.K / 32;
  if (!bf16) {
    CHECK(a.N % 64 == 0, "%s: f32 N %d", what, a.N);
    CHECK(a.S == 1, "%s: f32 split %d", what, a.S);
    t = {0, 16, 64, 1};
    return true;
  }
  if (mt > kMmTile && mt <= kMmTile + 8) {
    const int rt = mt - kMmTile;
    CHECK(rt == 2 || rt == 4 || rt == 8, "%s: RT %d", what, rt);
    const bool ok = (rt <= 4 && nt == 4) || nt == 2 || (rt >= 4 && nt == 12) ||
                    (rt >= 8 && (nt == 10 || nt == 18 || nt == 20));
    CHECK(ok, "%s: no medium-M instantiation for RT %d nt %d", what, rt, nt);
    const int cols = nt > 16 ? 8 * 16 * (nt - 16) : (nt > 8 ? 8 * 16 * (nt - 8) : 4 * 16 * nt);
    CHECK(a.S >= 1 && a.S <= KS, "%s: S %d of %d k-steps", what, a.S, KS);
    CHECK(a.N % cols == 0, "%s: N %d not a multiple of %d", what, a.N, cols);
    for (int g = 0; g < a.ngroups; ++g)
      CHECK(a.g[g].mrows >= 0 && a.g[g].mrows % 16 == 0 && a.g[g].mrows <= 16 * rt, "%s: mrows %d at RT %d",
            what, a.g[g].mrows, rt);
    t = {2, 16 * rt, cols, a.S};
    return true;
  }
  CHECK(mt >= kWgTile, "%s: unknown tile code %d", what, mt);
  const int m = mt - kWgTile;
  CHECK(m == 1 || m == 2 || m == 4, "%s: workgroup-tile rows %d", what, m);
  CHECK(nt == 4 || nt == 2 || (nt == 1 && epi == EPI_F32), "%s: workgroup-tile nt %d", what, nt);
  CHECK(a.ksteps % 4 == 0 && a.ksteps > 0, "%s: ksteps %d", what, a.ksteps);
  CHECK(a.ksteps * a.S == KS, "%s: %d splits of %d != %d k-steps", what, a.S, a.ksteps, KS);
  CHECK(a.N % (64 * nt) == 0, "%s: N %d nt %d", what, a.N, nt);
  t = {1, 16 * m, 64 * nt, a.S};
  return true;
}

// Replay the grid: every item through the kernel's own decode.
bool covers(const GemmArgs& a, const Tile& t, const char* what) {
  const int KS = a.K / 32;
  const int ncol = a.N / t.cols;
  int expect = 0;
  for (int k = 0; k < a.ngroups; ++k) {
    CHECK(a.g[k].item0 == expect, "%s: group %d item0 %d, expected %d", what, k, a.g[k].item0, expect);
    const int n_mc = a.g[k].n_mc;
    const int crows = (t.kind == 2 && a.g[k].mrows > 0) ? a.g[k].mrows : t.rows;
    CHECK(a.g[k].nrows >= 0, "%s: rows %d", what, a.g[k].nrows);
    CHECK((int64_t)n_mc * crows >= a.g[k].nrows && (n_mc == 0 || (int64_t)(n_mc - 1) * crows < a.g[k].nrows),
          "%s: group %d: %d chunks of %d rows for %d rows", what, k, n_mc, crows, a.g[k].nrows);
    expect += n_mc * ncol * t.S;
  }
  CHECK(a.total_items == expect, "%s: total %d, expected %d", what, a.total_items, expect);
  std::vector<std::vector<uint8_t>> hit(a.ngroups);
  for (int k = 0; k < a.ngroups; ++k) hit[k].assign((size_t)a.g[k].nrows * ncol * t.S, 0);
  for (int blk = 0; blk < a.total_items; ++blk) {
    int k = 0;
    for (int i = 1; i < kMaxGroups; ++i)
      if (i < a.ngroups && a.g[i].item0 <= blk) k = i;
    const GemmGroup& G = a.g[k];
    CHECK(G.n_mc > 0, "%s: item %d resolves to empty group %d", what, blk, k);
    const int idx = blk - G.item0;
    int mc, nb, s, crows;
    if (t.kind == 0) {
      mc = idx % G.n_mc; nb = idx / G.n_mc; s = 0; crows = 16;
    } else if (t.kind == 1) {
      mc = idx % G.n_mc; const int rest = idx / G.n_mc; s = rest % a.S; nb = rest / a.S; crows = t.rows;
    } else {
      mc = idx % G.n_mc; nb = (idx / G.n_mc) % ncol; s = idx / (G.n_mc * ncol);
      crows = G.mrows > 0 ? G.mrows : t.rows;
    }
    CHECK(nb < ncol && s < t.S, "%s: item %d: column block %d of %d, split %d of %d", what, blk, nb, ncol, s, t.S);
    const int rbase = G.row0 + mc * crows;
    const int rend = std::min(G.row0 + G.nrows, rbase + crows);
    CHECK(rbase < rend, "%s: item %d: empty row range", what, blk);
    for (int r = rbase; r < rend; ++r) {
      uint8_t& h = hit[k][((size_t)(r - G.row0) * ncol + nb) * t.S + s];
      CHECK(h == 0, "%s: row %d block %d split %d covered twice", what, r, nb, s);
      h = 1;
    }
  }
  for (int k = 0; k < a.ngroups; ++k)
    for (size_t i = 0; i < hit[k].size(); ++i)
      CHECK(hit[k][i] == 1, "%s: group %d cell %zu not covered", what, k, i);
  // the k-splits tile [0, KS)
  int kend = 0;
  for (int s = 0; s < t.S; ++s) {
    const int k0 = t.kind == 1 ? s * a.ksteps : (s * KS) / t.S;
    const int k1 = t.kind == 1 ? (s + 1) * a.ksteps : ((s + 1) * KS) / t.S;
    CHECK(k0 == kend && k1 > k0, "%s: split %d takes k-steps [%d, %d)", what, s, k0, k1);
    kend = k1;
  }
  CHECK(t.kind == 0 || kend == KS, "%s: splits end at %d of %d", what, kend, KS);
  return true;
}

bool check_case(const moa_engine& e, const Proj& p, const GemmPlanIn& in, const int* cut, int nshare) {
  char what[160];
  int totalM = 0;
  for (int g = 0; g < in.ngroups; ++g) totalM += in.nrows[g];
  std::snprintf(what, sizeof what, "%s %s K %d N %d, %d groups, %d rows", e.bf16 ? "bf16" : "f32", p.name, p.K,
                p.N, in.ngroups, totalM);
  float* part = reinterpret_cast<float*>(uintptr_t(1) << 20);   // never dereferenced
  GemmArgs whole;
  int mt = 0, nt = 0;
  bool large = false;
  plan_gemm(&e, in, 0, in.ngroups, p.K, p.N, p.epi, nullptr, 0, part, nullptr, 0, p.split, whole, mt, nt, large);
  Tile t;
  if (!dispatchable(e.bf16, whole, p.epi, mt, nt, t, what)) return false;
  if (!covers(whole, t, what)) return false;
  // the large-M plan: whole 128-row chunks on the three-stage 8-wave code
  // (medium gate-up at RT = 8 uses that code too, on smaller chunks)
  if (large) {
    CHECK(e.bf16 && mt == kMmTile + 8 && nt > 16, "%s: large plan on mt %d nt %d", what, mt, nt);
    for (int g = 0; g < whole.ngroups; ++g) CHECK(whole.g[g].mrows == 128, "%s: large chunk %d", what, whole.g[g].mrows);
  }
  if (!p.split) CHECK(whole.S == 1, "%s: unsplit projection split %d ways", what, whole.S);
  if (p.epi == EPI_SWIGLU && t.kind == 2 && !large)
    CHECK(whole.total_items <= 256, "%s: gate-up medium grid %d", what, whole.total_items);
  if (whole.S > 1) {
    CHECK(whole.out_split == (size_t)totalM * p.N, "%s: partial stride %zu", what, whole.out_split);
    CHECK((int64_t)whole.S * totalM * p.N <= e.lay.part_cap, "%s: %d partials of %d x %d exceed %lld floats", what,
          whole.S, totalM, p.N, (long long)e.lay.part_cap);
  }
  // share launches: contiguous group ranges planned from the whole step
  for (int u = 0; u < nshare; ++u) {
    const int g0 = cut[u], ng = cut[u + 1] - cut[u];
    if (ng == 0) continue;
    GemmArgs a;
    int smt = 0, snt = 0;
    bool slarge = false;
    plan_gemm(&e, in, g0, ng, p.K, p.N, p.epi, nullptr, 0, part, nullptr, 0, p.split, a, smt, snt, slarge);
    CHECK(smt == mt && snt == nt && slarge == large && a.S == whole.S && a.ksteps == whole.ksteps &&
              a.out_split == whole.out_split,
          "%s: share %d plans mt %d nt %d S %d, the step mt %d nt %d S %d", what, u, smt, snt, a.S, mt, nt, whole.S);
    for (int k = 0; k < ng; ++k)
      CHECK(a.g[k].row0 == whole.g[g0 + k].row0 && a.g[k].nrows == whole.g[g0 + k].nrows &&
                a.g[k].n_mc == whole.g[g0 + k].n_mc && a.g[k].mrows == whole.g[g0 + k].mrows &&
                a.g[k].W == in.W[g0 + k],
            "%s: share %d group %d differs from the step's plan", what, u, k);
    Tile ts;
    if (!dispatchable(e.bf16, a, p.epi, smt, snt, ts, what)) return false;
    if (!covers(a, ts, what)) return false;
  }
  return true;
}

// Large-M k-splits measured best on an MI355X (cold 8B weights, the GEMM
// plus its consumer's read of the partials), at the workspace of a
// 16,384-token prefill budget and 512 sequences: the fitted cost must keep
// choosing them.
bool measured_splits() {
  moa_engine_cfg cfg{};
  cfg.model = {32, 4096, 32, 8, 128, 14336, 128256, 500000.f, 1e-5f};
  cfg.dtype = MOA_BF16; cfg.kv_block_size = kBlock; cfg.num_kv_blocks = 4096; cfg.max_num_seqs = 512;
  cfg.max_prefill_tokens = 16384; cfg.max_model_len = 40000; cfg.max_models = 4;
  moa_engine e;
  e.cfg = cfg;
  e.bf16 = true;
  e.lay = make_layout(cfg);
  struct Case { const char* name; int K, N; std::vector<int> rows; int S; };
  const Case cases[] = {
      {"qkv", 4096, 6144, {512}, 5},          {"qkv", 4096, 6144, {300}, 7},
      {"qkv", 4096, 6144, {2048, 90, 80}, 1}, {"qkv", 4096, 6144, {700, 80, 90, 60}, 2},
      {"o", 4096, 4096, {2048, 90, 80}, 3},   {"o", 4096, 4096, {2600}, 3},
      {"o", 4096, 4096, {300}, 9},            {"o", 4096, 4096, {16384}, 1},
      {"down", 14336, 4096, {2048, 90, 80}, 5}, {"down", 14336, 4096, {300}, 10},
      {"down", 14336, 4096, {8000, 100, 90}, 3}, {"down", 14336, 4096, {16384}, 1},
  };
  for (const Case& c : cases) {
    GemmPlanIn in;
    in.ngroups = (int)c.rows.size();
    int row = 0;
    for (int g = 0; g < in.ngroups; ++g) { in.row0[g] = row; in.nrows[g] = c.rows[g]; row += c.rows[g]; in.W[g] = nullptr; }
    GemmArgs a;
    int mt = 0, nt = 0;
    bool large = false;
    plan_gemm(&e, in, 0, in.ngroups, c.K, c.N, EPI_F32, nullptr, 0, nullptr, nullptr, 0, true, a, mt, nt, large);
    CHECK(large && a.S == c.S, "%s at %d rows in %d groups: large %d S %d, measured best S %d", c.name, row, in.ngroups,
          large, a.S, c.S);
  }
  return true;
}

int rows_draw(int cap) {
  switch (rnd(6)) {
    case 0: return 0;
    case 1: return 1 + (int)rnd(16);
    case 2: return 17 + (int)rnd(48);
    case 3: return 65 + (int)rnd(191);
    case 4: return 256 + (int)rnd(std::max(1, cap - 256));
    default: return 1 + (int)rnd(std::max(1, cap));
  }
}

}  // namespace

int main(int argc, char** argv) {
  const int cases = argc > 1 ? std::atoi(argv[1]) : 400;
  if (argc > 2) g_rng ^= std::strtoull(argv[2], nullptr, 10) * 0x9e3779b97f4a7c15ull;   // another seed
  const Shape shapes[3] = {
      {"8B", {32, 4096, 32, 8, 128, 14336, 128256, 500000.f, 1e-5f}},
      {"1B", {16, 2048, 32, 8, 64, 8192, 128256, 500000.f, 1e-5f}},
      {"small", {2, 256, 8, 2, 64, 512, 1024, 10000.f, 1e-5f}},
  };
  const int prefill_caps[4] = {512, 2048, 8192, 16384};
  const int seq_caps[3] = {64, 256, 512};
  long planned = 0;
  if (!measured_splits()) return 1;
  for (int dt = 0; dt < 2; ++dt)
    for (const Shape& sh : shapes)
      for (int c = 0; c < cases; ++c) {
        moa_engine_cfg cfg{};
        cfg.model = sh.m;
        cfg.dtype = dt ? MOA_BF16 : MOA_F32;
        cfg.kv_block_size = kBlock;
        cfg.num_kv_blocks = 4096;
        cfg.max_num_seqs = seq_caps[rnd(3)];
        cfg.max_prefill_tokens = prefill_caps[rnd(4)];
        cfg.max_model_len = 40000;
        cfg.max_models = 1 + (int)rnd(kMaxModels);
        if (!valid_cfg(cfg)) { std::fprintf(stderr, "invalid config for %s\n", sh.name); return 1; }
        moa_engine e;
        e.cfg = cfg;
        e.bf16 = dt == 1;
        e.lay = make_layout(cfg);
        const moa_model_cfg& m = sh.m;
        const int qkv = (m.n_heads + 2 * m.n_kv_heads) * m.head_dim, qd = m.n_heads * m.head_dim;
        const Proj projs[5] = {
            {"qkv", m.d_model, qkv, EPI_F32, true, false},
            {"o", qd, m.d_model, EPI_F32, true, false},
            {"gate-up", m.d_model, 2 * m.ffn_dim, e.bf16 ? EPI_SWIGLU : EPI_F32, false, false},
            {"down", m.ffn_dim, m.d_model, EPI_F32, true, false},
            {"lm head", m.d_model, m.vocab, EPI_F32, false, true},
        };
        // a step's rows: up to max_models groups within the step's row cap
        GemmPlanIn in;
        in.ngroups = cfg.max_models;
        const int64_t tmax = e.lay.Tmax;
        int64_t total = 0;
        for (int g = 0; g < in.ngroups; ++g) {
          in.nrows[g] = rows_draw((int)std::min<int64_t>(tmax, 16384));
          total += in.nrows[g];
        }
        if (total > tmax)   // scale down to the step's cap
          for (int g = 0; g < in.ngroups; ++g) in.nrows[g] = (int)((int64_t)in.nrows[g] * tmax / total);
        int lm_rows[kMaxModels];
        int64_t lm_total = 0;
        for (int g = 0; g < in.ngroups; ++g) {
          lm_rows[g] = in.nrows[g] ? 1 + (int)rnd((uint32_t)std::min(in.nrows[g], cfg.max_num_seqs)) : 0;
          lm_total += lm_rows[g];
        }
        if (lm_total > cfg.max_num_seqs)
          for (int g = 0; g < in.ngroups; ++g) lm_rows[g] = (int)((int64_t)lm_rows[g] * cfg.max_num_seqs / lm_total);
        // model-stream shares: contiguous group ranges
        int nshare = 1 + (int)rnd(kMaxShares);
        int cut[kMaxShares + 1];
        cut[0] = 0;
        cut[nshare] = in.ngroups;
        for (int u = 1; u < nshare; ++u) cut[u] = std::max(cut[u - 1], (int)rnd((uint32_t)in.ngroups + 1));
        for (int u = 1; u < nshare; ++u) cut[u] = std::min(cut[u], in.ngroups);
        for (const Proj& p : projs) {
          GemmPlanIn pin = in;
          int row = 0;
          for (int g = 0; g < pin.ngroups; ++g) {
            if (p.lm) pin.nrows[g] = lm_rows[g];
            pin.row0[g] = row;
            row += pin.nrows[g];
            pin.W[g] = reinterpret_cast<const void*>(uintptr_t(g + 1) << 32);
          }
          if (row == 0) continue;
          if (!check_case(e, p, pin, cut, nshare)) continue;
          ++planned;
        }
      }
  if (g_fail) {
    std::fprintf(stderr, "gemm_plan_check: %d failures\n", g_fail);
    return 1;
  }
  std::printf("gemm_plan_check: ok (%ld plans)\n", planned);
  return 0;
}
