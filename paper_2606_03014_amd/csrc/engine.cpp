// Host side of the ragged MoA generation engine: request table, FIFO
// admission, paged-KV block allocator, step planner, metadata upload and the
// per-step kernel sequence. See include/moa.h for the contract.
#include "moa.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <deque>
#include <new>
#include <thread>
#include <vector>

#include "kernels.h"

using namespace moa;

namespace {

constexpr int kStageSlots = 4;    // steps that may be in flight (pinned staging ring)
constexpr int kTargetWaves = 4096;
constexpr int kBigMinRows = 256;    // a row group this large takes the large-M plan (128-row chunks)
constexpr int kBigTargetWgs = 256;  // one workgroup per CU
// Large-M k-split cost, fitted to cold-weight sweeps of the 8B projections
// (300 to 4,096 rows in one to four groups, S = 1..8; 4.6% rms): per
// 32-wide k-step of a workgroup, each round of the grid over the CUs costs
// kRoundUs and the grid's size in CU-fulls kGridUs; every byte of partial
// sums costs kPartialUs to write and, in the consumer, to read back.
constexpr double kRoundUs = 1.075, kGridUs = 0.442, kPartialUs = 0.37e-6;
// bf16 steps with several models run them on up to this many streams: the
// step's models are dealt out in shares of about equal cost (rows laid out
// share by share), the first on the caller's stream, the others on streams
// forked from it at the step's start and joined at its end, so one share's
// launch-bound kernels and grid tails overlap the others' work. Two is the measured best on the 4x1B batch: 19.9k tok/s
// on one stream, 20.8k on two, 19.7k on three, 14.2k on four with shares by
// model index (more streams than the process's hardware queues serialise);
// with cost-balanced shares 21.4k on two and 20.8k on three.
constexpr int kModelStreams = 2;
constexpr int kMaxShares = 4;
static_assert(kModelStreams >= 1 && kModelStreams <= kMaxShares, "model streams");

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct Request {
  int64_t id = 0;
  int32_t model = 0, P = 0, G = 0, need = 0;
  // Injected history: positions 0..shift-1 arrive as K/V, the seed token sits
  // at position shift (P = shift + 1) and token-store slot tok_off holds it.
  // Position p's token lives at slot tok_off + p - shift.
  int32_t shift = 0;
  bool history = false;
  std::vector<char> host_kv;          // caller's K/V until admission (empty: device fill)
  int32_t pre = 0, gen = 0;
  bool fresh = false;
  int64_t tok_off = -1;               // token store: P prompt slots, then G outputs
  int64_t bt_off = -1;                // block store: need entries
  std::vector<int32_t> blocks;
  std::vector<int32_t> prompt;        // host copy until uploaded at admission
  int64_t admit_step = -1, finish_step = -1;
  std::vector<std::array<int64_t, 3>> chunks;
  int state = 0;                      // 0 pending, 1 running, 2 retired, 3 collected
  float* capture = nullptr;
};

struct ModelDev {
  // device pointers (bf16 bits or f32)
  const void* embed = nullptr;
  std::vector<const void*> attn_norm, wqkv, wo, mlp_norm, wgu, wdown;
  const void* final_norm = nullptr;
  const void* lm_head = nullptr;
};

// Free-block set: bit i set <=> block i free. take() returns the k smallest.
struct BlockSet {
  std::vector<uint64_t> bits;
  int64_t nfree = 0;
  size_t lo = 0;   // no free bit below word lo
  void init(int64_t n) {
    bits.assign((n + 63) / 64, 0);
    for (int64_t i = 0; i < n; ++i) bits[i >> 6] |= 1ull << (i & 63);
    nfree = n;
    lo = 0;
  }
  void take(int32_t k, std::vector<int32_t>& out) {
    out.clear();
    out.reserve(k);
    size_t w = lo;
    while ((int32_t)out.size() < k) {
      uint64_t v = bits[w];
      while (v && (int32_t)out.size() < k) {
        int b = __builtin_ctzll(v);
        v &= v - 1;
        out.push_back((int32_t)(w * 64 + b));
      }
      if ((int32_t)out.size() < k) ++w;
    }
    for (int32_t b : out) bits[b >> 6] &= ~(1ull << (b & 63));
    nfree -= k;
    while (lo < bits.size() && bits[lo] == 0) ++lo;
  }
  void give(const std::vector<int32_t>& v) {
    for (int32_t b : v) {
      bits[b >> 6] |= 1ull << (b & 63);
      if ((size_t)(b >> 6) < lo) lo = b >> 6;
    }
    nfree += (int64_t)v.size();
  }
};

struct Layout {
  size_t esz;
  int64_t Tmax, Rmax, slots_cap, items_cap, red_cap, part_cap;
  size_t model_bytes, kv_bytes, block_bytes;
  size_t off_xpart[kMaxShares - 1];   // split-K partials of shares 1.. (0: none)
  size_t off_kv, off_tok, off_bt, off_rope, off_meta, off_x, off_xn, off_part, off_q, off_ao, off_h,
      off_logits, off_xl, off_pacc, off_pml, off_models, total;
  int64_t token_store, block_store, meta_ints;
};

bool valid_cfg(const moa_engine_cfg& c) {
  const moa_model_cfg& m = c.model;
  if (c.dtype != MOA_F32 && c.dtype != MOA_BF16) return false;
  if (c.kv_block_size != kBlock) return false;
  if (m.n_layers < 1 || m.d_model < 32 || m.n_heads < 1 || m.n_kv_heads < 1 || m.vocab < 1 || m.ffn_dim < 32)
    return false;
  if (m.n_heads % m.n_kv_heads) return false;
  const int gq = m.n_heads / m.n_kv_heads;
  if (gq != 1 && gq != 2 && gq != 4 && gq != 8) return false;
  if (m.head_dim != 64 && m.head_dim != 128) return false;
  if (!(m.rms_eps > 0.f) || !(m.rope_theta > 0.f)) return false;
  if (m.d_model % 256 || m.d_model > 4096 || m.ffn_dim % 64 || m.vocab % 16) return false;
  if (c.dtype == MOA_F32 && (m.vocab % 64 || (2 * m.ffn_dim) % 64)) return false;
  // bf16 GEMMs stream K in batches of 4 MFMA k-steps of 32, and every
  // projection width (qkv, gate-up, LM head) is a whole number of 128-column
  // workgroup tiles
  if (c.dtype == MOA_BF16 && (m.d_model % 128 || m.ffn_dim % 128 || (m.n_heads * m.head_dim) % 128 ||
                              ((m.n_heads + 2 * m.n_kv_heads) * m.head_dim) % 128 || m.vocab % 128))
    return false;
  if (c.num_kv_blocks < 1 || c.max_num_seqs < 1 || c.max_prefill_tokens < 0 || c.max_model_len < 2) return false;
  if (c.max_models < 1 || c.max_models > kMaxModels) return false;
  if (c.token_store < 0 || c.block_store < 0) return false;
  return true;
}

Layout make_layout(const moa_engine_cfg& c) {
  Layout L{};
  const moa_model_cfg& m = c.model;
  L.esz = c.dtype == MOA_BF16 ? 2 : 4;
  const int64_t d = m.d_model, hd = m.head_dim, nh = m.n_heads, nkv = m.n_kv_heads, V = m.vocab,
                F = m.ffn_dim, Lr = m.n_layers;
  const int64_t qkv = (nh + 2 * nkv) * hd;
  L.Tmax = (int64_t)c.max_prefill_tokens + c.max_num_seqs;
  L.Rmax = c.max_num_seqs;
  L.slots_cap = (int64_t)c.num_kv_blocks * kBlock / kSplitKeys + c.max_num_seqs + 1;
  L.items_cap = L.Tmax + L.slots_cap;
  L.red_cap = c.max_num_seqs;
  // split-K partials: a prefill-sized step unsplit, or a full decode batch
  // split up to 8 ways (a few hundred rows need the split to fill the CUs)
  int64_t pc = std::max(L.Tmax, (int64_t)8 * c.max_num_seqs) * std::max(qkv, d);
  if (c.dtype == MOA_F32) pc = std::max(pc, L.Tmax * 2 * F);
  L.part_cap = pc;
  L.token_store = c.token_store ? c.token_store : (int64_t)64 << 20;
  L.block_store = c.block_store ? c.block_store : (int64_t)16 << 20;
  L.meta_ints = 4 * L.Tmax + 2 * L.Rmax + 8 * L.items_cap + 4 * L.red_cap + 4 * L.Tmax;
  L.block_bytes = (size_t)Lr * nkv * 2 * kBlock * hd * L.esz;
  L.kv_bytes = L.block_bytes * (size_t)c.num_kv_blocks;
  const size_t per_layer = (size_t)(2 * d + qkv * d + d * nh * hd + 3 * F * d) * L.esz;
  L.model_bytes = align_up((size_t)(2 * V * d + d) * L.esz + 256 * (8 + 6 * Lr) + per_layer * Lr, 256);

  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes, 256); return o; };
  L.off_kv = take(L.kv_bytes);
  L.off_tok = take((size_t)L.token_store * 4);
  L.off_bt = take((size_t)L.block_store * 4);
  L.off_rope = take((size_t)c.max_model_len * (hd / 2) * sizeof(float2));
  L.off_meta = take((size_t)L.meta_ints * 4);
  L.off_x = take((size_t)L.Tmax * d * 4);
  // GEMM inputs (xn, ao, h) hold two planes: bf16 hi and lo (fp32 mode uses the first)
  L.off_xn = take((size_t)2 * L.Tmax * d * L.esz);
  L.off_part = take((size_t)L.part_cap * 4);
  // every further share's own split-K partials (its projections run while
  // another share's, of another width, are in flight)
  const int nx = (c.dtype == MOA_BF16 && !(c.flags & MOA_FLAG_ONE_STREAM))
                     ? std::min(kModelStreams, (int)c.max_models) - 1 : 0;
  for (int k = 0; k < kMaxShares - 1; ++k) L.off_xpart[k] = k < nx ? take((size_t)L.part_cap * 4) : 0;
  L.off_q = take((size_t)L.Tmax * nh * hd * 4);
  L.off_ao = take((size_t)2 * L.Tmax * nh * hd * L.esz);
  L.off_h = take((size_t)2 * L.Tmax * F * L.esz);
  L.off_logits = take((size_t)L.Rmax * V * 4);
  // LM-head input (final-norm output in LM-row order; split pair in bf16)
  L.off_xl = take((size_t)2 * L.Rmax * d * L.esz);
  L.off_pacc = take((size_t)L.slots_cap * nh * hd * 4);
  L.off_pml = take((size_t)L.slots_cap * nh * 2 * 4);
  L.off_models = off;
  L.total = off + L.model_bytes * (size_t)c.max_models;
  return L;
}

}  // namespace

struct moa_engine {
  moa_engine_cfg cfg{};
  Layout lay{};
  bool plan_only = false;
  bool bf16 = false;
  bool broken = false;
  hipStream_t stream = nullptr;
  hipStream_t copy_stream = nullptr;
  int nstreams = 1;                   // model streams: the caller's + xs[0 .. nstreams - 2]
  hipStream_t xs[kMaxShares - 1] = {};
  hipEvent_t ev_fork = nullptr;
  hipEvent_t ev_join[kMaxShares - 1] = {};
  char* arena = nullptr;
  size_t arena_bytes = 0;
  size_t model_top = 0;

  std::vector<ModelDev> models;
  std::vector<Request> reqs;
  std::deque<int64_t> pending;
  std::vector<int64_t> running;
  std::vector<int64_t> done;          // retired, not collected, in retirement order
  BlockSet free_blocks;
  int64_t tok_top = 0, bt_top = 0;
  int64_t step_idx = 0;
  int64_t live = 0;                   // requests not yet collected
  std::vector<std::array<int64_t, 6>> trace;

  // device views
  char* kv = nullptr;
  int* tok_store = nullptr;
  int* bt_store = nullptr;
  float2* rope = nullptr;
  int* meta = nullptr;
  float* x = nullptr;
  void* xn = nullptr;
  float* part = nullptr;
  float* xpart[kMaxShares - 1] = {};  // partials of shares 1..
  float* q = nullptr;
  void* ao = nullptr;
  void* h = nullptr;
  float* logits = nullptr;
  void* xl = nullptr;                 // LM-head input rows (final norm output)
  float* pacc = nullptr;
  float* pml = nullptr;
  void* scratch = nullptr;            // this GPU's library scratch array (moa_step_noalloc)

  // pinned staging ring and per-step completion events
  struct Stage { char* buf = nullptr; size_t cap = 0; };
  Stage stage[kStageSlots];
  hipEvent_t ev[kStageSlots] = {};
  int64_t ev_step[kStageSlots] = {-1, -1, -1, -1};
  int32_t* pinned_out = nullptr;
  size_t pinned_out_cap = 0;
  // host prompt copies an allocation-free step uploads straight from, kept
  // until the step that read them completes (released when its slot is reused)
  std::vector<std::vector<int32_t>> keepalive[kStageSlots];

  // kernel timing (inspection hook): event pairs around launches of sampled steps
  struct Timed { int cls, cls2; hipEvent_t a, b; double bytes, flops; };
  int time_every = 0;
  bool time_now = false;
  bool account = false;
  double peak_bw = 8e12, peak_flops = 2.5e15;
  std::vector<hipEvent_t> ev_pool;
  std::vector<Timed> timed;
  moa_kernel_stats kstats[MOA_K_COUNT] = {};

  // per-step host plan (reused vectors)
  std::vector<int> r_tok, r_pos, r_bt, r_model, l_src, l_dst;
  std::vector<AttnItem> items;
  std::vector<ReduceItem> red;
  std::vector<PrefillItem> pitems;
  // the step's shares: share u holds model groups [sh_group[u], sh_group[u+1]),
  // rows, LM rows and attention / combine / prefill items likewise (each item
  // list sorted by share first)
  int morder[kMaxModels] = {};        // model order of the step's rows
  int nactive = 0;                    // models with rows (the first nactive of morder)
  double mcost[kMaxModels] = {};      // the split's cost per model
  int nshare = 1;
  int sh_group[kMaxShares + 1] = {}, sh_row[kMaxShares + 1] = {}, sh_lm[kMaxShares + 1] = {};
  int sh_item[kMaxShares + 1] = {}, sh_red[kMaxShares + 1] = {}, sh_pre[kMaxShares + 1] = {};
};

namespace {

moa_status hip_fail(moa_engine* e, hipError_t err, const char* what) {
  if (e) e->broken = true;
  std::fprintf(stderr, "moa: HIP error in %s: %s\n", what, hipGetErrorString(err));
  return MOA_EHIP;
}

#define HIPCHK(call, what)                              \
  do {                                                  \
    hipError_t _err = (call);                           \
    if (_err != hipSuccess) return hip_fail(e, _err, what); \
  } while (0)

hipEvent_t pool_event(moa_engine* e) {
  if (!e->ev_pool.empty()) {
    hipEvent_t v = e->ev_pool.back();
    e->ev_pool.pop_back();
    return v;
  }
  hipEvent_t v = nullptr;
  if (hipEventCreate(&v) != hipSuccess) return nullptr;
  return v;
}

// Fold finished timing pairs into the statistics (waits for each pair).
moa_status resolve_timed(moa_engine* e) {
  for (auto& t : e->timed) {
    HIPCHK(hipEventSynchronize(t.b), "timing wait");
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, t.a, t.b) != hipSuccess) {   // launch carried no work
      (void)hipGetLastError();
      e->ev_pool.push_back(t.a);
      e->ev_pool.push_back(t.b);
      continue;
    }
    for (int c : {t.cls, t.cls2}) {
      if (c < 0) continue;
      moa_kernel_stats& k = e->kstats[c];
      k.launches += 1;
      k.ms += ms;
      k.bytes += t.bytes;
      k.flops += t.flops;
    }
    e->ev_pool.push_back(t.a);
    e->ev_pool.push_back(t.b);
  }
  e->timed.clear();
  return MOA_OK;
}

// Launch `call` (an expression yielding hipError_t). Every launch is
// accounted (algorithmic bytes, flops, roofline time) under class `cls` and,
// when cls2 >= 0, under the view class cls2 too; in sampled steps the
// kernel's own dispatch also carries a start/stop event pair.
#define LAUNCH2(cls, cls2, bytes_, flops_, call, what)                            \
  do {                                                                           \
    if (e->account) {                                                            \
      const double _by = (double)(bytes_), _fl = (double)(flops_);               \
      for (int _c : {(int)(cls), (int)(cls2)}) {                                 \
        if (_c < 0) continue;                                                    \
        moa_kernel_stats& _k = e->kstats[_c];                                    \
        _k.launches_all += 1;                                                    \
        _k.bytes_all += _by;                                                     \
        _k.flops_all += _fl;                                                     \
        _k.roof_ms_all += 1e3 * std::max(_by / e->peak_bw, _fl / e->peak_flops); \
      }                                                                          \
    }                                                                            \
    if (e->time_now) {                                                           \
      hipEvent_t _a = pool_event(e), _b = pool_event(e);                         \
      if (!_a || !_b) return hip_fail(e, hipErrorOutOfMemory, "timing events");  \
      set_launch_events(_a, _b);                                                 \
      hipError_t _err = (call);                                                  \
      set_launch_events(nullptr, nullptr);                                       \
      if (_err != hipSuccess) return hip_fail(e, _err, what);                    \
      e->timed.push_back({(cls), (cls2), _a, _b, (double)(bytes_), (double)(flops_)}); \
    } else {                                                                     \
      HIPCHK((call), what);                                                      \
    }                                                                            \
  } while (0)
#define LAUNCH(cls, bytes_, flops_, call, what) LAUNCH2(cls, -1, bytes_, flops_, call, what)
// a GEMM launch: its projection class plus the view of the kernel that runs it
#define LAUNCH_GEMM(cls, large_, bytes_, flops_, call, what) \
  LAUNCH2(cls, (large_) ? MOA_K_GEMM_LARGE_M : MOA_K_GEMM_SMALL_M, bytes_, flops_, call, what)

// Tile-shuffle a row-major [N][K] bf16 matrix into MFMA B-fragment order:
// fragment (n/16, k/32) is 64 lanes x 8 contiguous elements, lane = n%16 +
// 16*((k%32)/8). Rows are taken from src_rows(n) so the gate/up interleave and
// the q|k|v concatenation are done in the same pass.
template <class RowFn>
void shuffle_bf16(uint16_t* dst, int64_t N, int64_t K, RowFn src_row) {
  const int64_t KS = K / 32, NT = N / 16;
  auto work = [&](int64_t t0, int64_t t1) {
    for (int64_t nt = t0; nt < t1; ++nt)
      for (int r = 0; r < 16; ++r) {
        const uint16_t* s = src_row(nt * 16 + r);
        for (int64_t k = 0; k < K; ++k) {
          const int64_t ks = k >> 5, kk = k & 31;
          dst[((nt * KS + ks) * 64 + (r + 16 * (kk >> 3))) * 8 + (kk & 7)] = s[k];
        }
      }
  };
  unsigned nth = std::max(1u, std::min(16u, std::thread::hardware_concurrency()));
  if (NT < 64) nth = 1;
  std::vector<std::thread> th;
  for (unsigned i = 0; i < nth; ++i) th.emplace_back(work, NT * i / nth, NT * (i + 1) / nth);
  for (auto& t : th) t.join();
}

struct GemmPlanIn {
  int ngroups = 0;
  int row0[kMaxModels], nrows[kMaxModels];
  const void* W[kMaxModels];
};

// Choose the tiling and k-split of one grouped GEMM and fill its arguments.
// X is a split-bf16 pair (lo plane x_lo elements after hi) in bf16 mode.
// Tile, split and partial stride are chosen from every group of `in` (the
// whole step, so a launch that carries only the groups [g0, g0 + ng) plans
// the same way and writes its partials where the consumer of the whole step
// expects them); the arguments carry only those groups.
// A step sampled for kernel timing (one in time_every; never an
// allocation-free step) runs every kernel on the caller's stream, so each
// timed launch carries the whole step and no other stream's kernels run
// beside it: its duration is its own.
bool step_is_timed(const moa_engine* e, bool noalloc) {
  return !noalloc && e->time_every > 0 && (e->step_idx % e->time_every) == 0;
}

void plan_gemm(const moa_engine* e, const GemmPlanIn& in, int g0, int ng, int K, int N, int epi, const void* X,
               size_t x_lo, float* out, uint16_t* hout, size_t h_lo, bool allow_split, GemmArgs& a, int& mt,
               int& nt, bool& large) {
  std::memset(&a, 0, sizeof(a));
  large = false;
  a.ngroups = ng;
  a.X = X;
  a.x_lo = x_lo;
  a.h_lo = h_lo;
  a.K = K;
  a.N = N;
  a.out = out;
  a.hout = hout;
  int maxM = 0, totalM = 0;
  for (int g = 0; g < in.ngroups; ++g) { maxM = std::max(maxM, in.nrows[g]); totalM += in.nrows[g]; }
  if (!e->bf16) {
    mt = 1; nt = 1;
    int item = 0;
    for (int k = 0; k < ng; ++k) {
      const int g = g0 + k;
      a.g[k].W = in.W[g]; a.g[k].row0 = in.row0[g]; a.g[k].nrows = in.nrows[g];
      a.g[k].n_mc = (in.nrows[g] + 15) / 16;
      a.g[k].item0 = item;
      item += a.g[k].n_mc * (N / 64);
    }
    a.S = 1; a.ksteps = 0; a.out_split = 0; a.total_items = item;
    return;
  }
  const int KS = K / 32;
  // The large-M plan (whole 128-row chunks, split-K only to fill the CUs)
  // from 256 rows in any group, and below that where every non-empty group
  // has enough rows for a long k run per workgroup to amortise its set-up:
  // square and deep-K projections (N <= K) from 160 rows, wide ones with
  // K >= 4096 from 192 (thresholds from cold-weight sweeps of both model
  // widths, one and four equal groups, measured with the 128-row tiles).
  const int big_min = N <= K ? 160 : (K >= 4096 ? 192 : kBigMinRows);
  int minM = maxM;
  for (int g = 0; g < in.ngroups; ++g)
    if (in.nrows[g] > 0) minM = std::min(minM, in.nrows[g]);
  if ((maxM >= kBigMinRows || minM >= big_min) && N % 256 == 0) {
    // matrix-core bound: the medium-M kernel on whole 128-row chunks, 8
    // waves over 512 columns (256 where N is not a multiple of 512) with a
    // three-stage weight ring.
    // Measured against a 32x32-MFMA kernel that staged both operands in LDS
    // (128 x 512 tiles): 3-29% faster from 512 to 16k rows on 8B shapes, and
    // more where small groups share the launch (no padded rows multiplied).
    large = true;
    const int ct = N % 512 == 0 ? 4 : 2;
    mt = kMmTile + 8;
    nt = 16 + ct;
    const int ncol = N / (128 * ct);
    int base = 0;
    for (int g = 0; g < in.ngroups; ++g) base += ((in.nrows[g] + 127) / 128) * ncol;
    // k-split (any S; at least 8 k-steps each) at the least fitted cost: a
    // grid just past the CUs runs a second, nearly empty round, and every
    // split adds partial sums. Against a power-of-two split grown until the
    // grid covered the CUs, measured with the consumer's read: o and down
    // 15-30% faster at 300-2,200 rows in several groups (S = 3..7 where
    // that gave 2 or 4), qkv 7-28% (S = 1 or 2 against 2 or 4; 5 against 8
    // at 512 rows in one group).
    int S = 1;
    if (allow_split) {
      double best = 0;
      for (int s = 1; s <= 16 && KS / s >= 8; ++s) {
        if ((int64_t)s * totalM * N > e->lay.part_cap) break;
        const double items = (double)base * s;
        const double cost = (kRoundUs * std::ceil(items / kBigTargetWgs) + kGridUs * items / kBigTargetWgs) * KS / s +
                            kPartialUs * 4.0 * s * (double)totalM * N;
        if (s == 1 || cost < best) { best = cost; S = s; }
      }
    }
    a.S = S;
    a.ksteps = KS / S;                     // informational: split s takes k-steps [s*KS/S, (s+1)*KS/S)
    a.out_split = (size_t)totalM * N;
    int item = 0;
    for (int k = 0; k < ng; ++k) {
      const int g = g0 + k;
      a.g[k].W = in.W[g]; a.g[k].row0 = in.row0[g]; a.g[k].nrows = in.nrows[g];
      a.g[k].mrows = 128;
      a.g[k].n_mc = (in.nrows[g] + 127) / 128;
      a.g[k].item0 = item;
      item += a.g[k].n_mc * S * ncol;
    }
    a.total_items = item;
    return;
  }
  // Medium row counts (17 and up per model, below the large-M thresholds):
  // the medium-M kernel.
  //  * Whole 16-row tiles of a group per workgroup: RT tiles per row chunk,
  //    2 up to 32 rows, 4 up to 64, else 8.
  //  * 8 waves over 512 columns where N allows; otherwise 8 waves over 256
  //    at RT = 8 and 4 waves over 256 below (a vocabulary of 128,256 is
  //    501 x 256, and two 64-row chunks per model would stream its LM head
  //    twice).
  //  * About one workgroup per CU. F32 projections take the k-split that
  //    brings the grid nearest ~224 workgroups; gate-up (no k-split: its
  //    SwiGLU epilogue needs the whole sum) takes the first tile shape whose
  //    grid has 150..256 workgroups, else the workgroup-tile kernel.
  // Measured on 8B shapes with cold weights, three groups of 16..200 rows:
  // 2-40% faster per projection than the workgroup-tile kernel, and
  // bit-identical on the same split. A 4-wave, 64-row-chunk plan with
  // three k-splits for the square O projection (its norm then reads fewer
  // partials) measured no faster in the 3+1x8B window.
  if (maxM > 16 && N % 256 == 0) {
    struct Shape { int rt, nw, ct; };
    auto chunks_of = [&](int rt) {
      int c = 0;
      for (int g = 0; g < in.ngroups; ++g) c += (in.nrows[g] + 16 * rt - 1) / (16 * rt);
      return c;
    };
    const int rt0 = maxM <= 32 ? 2 : (maxM <= 64 ? 4 : 8);
    Shape sh{0, 0, 0};
    int S = 1;
    if (epi == EPI_SWIGLU) {
      const int rtb = std::max(rt0, 4);
      const Shape cand[4] = {{rtb, 8, 4}, {rtb == 8 ? 8 : 0, 8, 2}, {4, 4, 4}, {2, 4, 4}};
      for (const Shape& c : cand) {
        if (c.rt == 0 || N % (16 * c.nw * c.ct)) continue;
        const int items = chunks_of(c.rt) * (N / (16 * c.nw * c.ct));
        if (items >= 150 && items <= 256) { sh = c; break; }
      }
    } else {
      sh = (rt0 >= 4 && N % 512 == 0) ? Shape{rt0, 8, 4} : (rt0 == 8 ? Shape{8, 8, 2} : Shape{rt0, 4, 4});
      if (allow_split) {
        const int base = chunks_of(sh.rt) * (N / (16 * sh.nw * sh.ct));
        S = std::max(1, std::min(16, (224 + base / 2) / std::max(base, 1)));
        while (S > 1 && ((int64_t)S * totalM * N > e->lay.part_cap || S > KS)) --S;
      }
    }
    if (sh.rt) {
      const int ncol = N / (16 * sh.nw * sh.ct);
      // Row chunks of up to T 16-row tiles per group. Gate-up (one k-split)
      // takes the smallest T, down to 4, whose grid still fits 256
      // workgroups: a large group's rows then spread over more workgroups
      // (its split-bf16 MFMA work, not the weight stream, is what holds the
      // others up from ~5 tiles per workgroup), and the chunks of one weight
      // column block run side by side on one XCD, which reads it once. The
      // k-split of the other projections already divides every workgroup.
      auto tiles = [&](int g) { return (in.nrows[g] + 15) / 16; };
      int T = sh.rt;
      if (epi == EPI_SWIGLU)
        for (int t = sh.rt - 1; t >= 4; --t) {
          int items = 0;
          for (int g = 0; g < in.ngroups; ++g) items += (tiles(g) + t - 1) / t * ncol;
          if (items > 256) break;
          T = t;
        }
      mt = kMmTile + sh.rt;
      // 8 waves: gate-up at RT = 8 with the three-stage weight ring (1-2%
      // faster there; the F32 projections' shorter k-splits prefer two)
      nt = sh.nw == 8 ? (epi == EPI_SWIGLU && sh.rt == 8 ? 16 : 8) + sh.ct : sh.ct;
      a.S = S;
      a.ksteps = KS / S;                   // informational: split s takes k-steps [s*KS/S, (s+1)*KS/S)
      a.out_split = (size_t)totalM * N;
      int item = 0;
      for (int k = 0; k < ng; ++k) {
        const int g = g0 + k;
        a.g[k].W = in.W[g]; a.g[k].row0 = in.row0[g]; a.g[k].nrows = in.nrows[g];
        const int tg = std::max(1, tiles(g));
        const int nch = (tg + T - 1) / T;
        a.g[k].mrows = 16 * ((tg + nch - 1) / nch);          // balanced chunks of at most T tiles
        a.g[k].n_mc = (in.nrows[g] + a.g[k].mrows - 1) / a.g[k].mrows;   // 0 for an empty group
        a.g[k].item0 = item;
        item += a.g[k].n_mc * S * ncol;
      }
      a.total_items = item;
      return;
    }
  }
  const int wmt = maxM <= 16 ? 1 : (maxM <= 32 ? 2 : 4);
  const int wnt = (maxM > 64 && N % 256 == 0) ? 4 : 2;
  // workgroup items: 16*wmt rows x 64*wnt columns (every bf16 projection
  // width is a multiple of 128: moa_create checks it)
  mt = kWgTile + wmt;
  nt = wnt;
  const int tiles = N / (64 * wnt);
  const int rows_per = 16 * wmt;
  int target = kTargetWaves / 4, base = 0;
  for (int g = 0; g < in.ngroups; ++g) base += ((in.nrows[g] + rows_per - 1) / rows_per) * tiles;
  // split-K granularity and target, from weight-streaming sweeps with cold
  // weights: deep-K projections (K >= 4N) stream best with half the
  // workgroups (longer k runs per workgroup); square ones at <= 8 rows with
  // twice as many (k runs of 4 stages)
  int kmul = 8;
  if (K >= 4 * N) target /= 2;
  else if (K == N && maxM <= 8) { target *= 2; kmul = 4; }
  int S = 1;
  if (allow_split) {
    while (base * S < target && KS % (S * 2 * kmul) == 0 &&
           (int64_t)S * 2 * totalM * N <= e->lay.part_cap && S < 16)
      S *= 2;
  }
  a.S = S;
  a.ksteps = KS / S;
  a.out_split = (size_t)totalM * N;  // partial s lives at out + s * rows * N
  int item = 0;
  for (int k = 0; k < ng; ++k) {
    const int g = g0 + k;
    a.g[k].W = in.W[g]; a.g[k].row0 = in.row0[g]; a.g[k].nrows = in.nrows[g];
    a.g[k].n_mc = (in.nrows[g] + rows_per - 1) / rows_per;
    a.g[k].item0 = item;
    item += a.g[k].n_mc * S * tiles;
  }
  a.total_items = item;
}

}  // namespace

// ==================================================================== C ABI

extern "C" {

const char* moa_status_str(moa_status s) {
  switch (s) {
    case MOA_OK: return "MOA_OK";
    case MOA_EINVAL: return "MOA_EINVAL: invalid argument";
    case MOA_ENOMEM: return "MOA_ENOMEM: arena or store too small";
    case MOA_ENOSPC: return "MOA_ENOSPC: request can never fit the KV pool";
    case MOA_ESTATE: return "MOA_ESTATE: call not valid in this state";
    case MOA_EHIP: return "MOA_EHIP: HIP runtime error";
  }
  return "unknown moa_status";
}

moa_status moa_arena_bytes(const moa_engine_cfg* cfg, size_t* bytes) {
  if (!cfg || !bytes || !valid_cfg(*cfg)) return MOA_EINVAL;
  *bytes = make_layout(*cfg).total;
  return MOA_OK;
}

moa_status moa_create(const moa_engine_cfg* cfg, void* dev_arena, size_t arena_bytes, void* hip_stream,
                      moa_engine** out) {
  if (!cfg || !out || !valid_cfg(*cfg)) return MOA_EINVAL;
  *out = nullptr;
  const bool plan_only = (cfg->flags & MOA_FLAG_PLAN_ONLY) != 0;
  Layout L = make_layout(*cfg);
  if (!plan_only) {
    if (!dev_arena) return MOA_EINVAL;
    if (arena_bytes < L.total) return MOA_ENOMEM;
    if (((uintptr_t)dev_arena) % 256) return MOA_EINVAL;
  }
  moa_engine* e = new (std::nothrow) moa_engine();
  if (!e) return MOA_ENOMEM;
  e->cfg = *cfg;
  e->lay = L;
  e->plan_only = plan_only;
  e->bf16 = cfg->dtype == MOA_BF16;
  e->free_blocks.init(cfg->num_kv_blocks);
  e->model_top = L.off_models;
  // a dry run plans the model-stream shares a GPU engine would use
  if (plan_only && L.off_xpart[0]) e->nstreams = 1 + (int)std::count_if(L.off_xpart, L.off_xpart + (kMaxShares - 1), [](size_t o) { return o != 0; });
  if (!plan_only) {
    e->stream = (hipStream_t)hip_stream;
    e->arena = (char*)dev_arena;
    e->arena_bytes = arena_bytes;
    char* A = e->arena;
    e->kv = A + L.off_kv;
    e->tok_store = (int*)(A + L.off_tok);
    e->bt_store = (int*)(A + L.off_bt);
    e->rope = (float2*)(A + L.off_rope);
    e->meta = (int*)(A + L.off_meta);
    e->x = (float*)(A + L.off_x);
    e->xn = A + L.off_xn;
    e->part = (float*)(A + L.off_part);
    for (int k = 0; k < kMaxShares - 1; ++k) e->xpart[k] = L.off_xpart[k] ? (float*)(A + L.off_xpart[k]) : nullptr;
    e->q = (float*)(A + L.off_q);
    e->ao = A + L.off_ao;
    e->h = A + L.off_h;
    e->logits = (float*)(A + L.off_logits);
    e->xl = A + L.off_xl;
    e->pacc = (float*)(A + L.off_pacc);
    e->pml = (float*)(A + L.off_pml);
    hipError_t err = hipStreamCreateWithFlags(&e->copy_stream, hipStreamNonBlocking);
    for (int i = 0; i < kStageSlots && err == hipSuccess; ++i) err = hipEventCreateWithFlags(&e->ev[i], hipEventDisableTiming);
    if (err == hipSuccess && e->xpart[0]) err = hipEventCreateWithFlags(&e->ev_fork, hipEventDisableTiming);
    for (int k = 0; k < kMaxShares - 1 && err == hipSuccess && e->xpart[k]; ++k) {
      err = hipStreamCreateWithFlags(&e->xs[k], hipStreamNonBlocking);
      if (err == hipSuccess) err = hipEventCreateWithFlags(&e->ev_join[k], hipEventDisableTiming);
      if (err == hipSuccess) e->nstreams = k + 2;
    }
    if (err == hipSuccess) {
      // RoPE table: angle pos * theta^(-2i/hd) and its cos/sin in double, stored as fp32.
      const int hd = cfg->model.head_dim, half = hd / 2;
      std::vector<float2> tab((size_t)cfg->max_model_len * half);
      for (int p = 0; p < cfg->max_model_len; ++p)
        for (int i = 0; i < half; ++i) {
          const double inv = std::pow((double)cfg->model.rope_theta, -(2.0 * i) / hd);
          const double ang = (double)p * inv;
          tab[(size_t)p * half + i] = make_float2((float)std::cos(ang), (float)std::sin(ang));
        }
      err = hipMemcpy(e->rope, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice);
    }
    if (err == hipSuccess) err = scratch_address(&e->scratch);
    // staging slots hold the largest step metadata from the start, so an
    // allocation-free step never has to grow them
    for (int i = 0; i < kStageSlots && err == hipSuccess; ++i) {
      const size_t cap = std::max((size_t)L.meta_ints * 4, (size_t)1 << 20);
      err = hipHostMalloc((void**)&e->stage[i].buf, cap, hipHostMallocDefault);
      if (err == hipSuccess) e->stage[i].cap = cap;
    }
    if (err != hipSuccess) {
      hip_fail(nullptr, err, "moa_create");
      moa_destroy(e);
      return MOA_EHIP;
    }
  }
  *out = e;
  return MOA_OK;
}

void moa_destroy(moa_engine* e) {
  if (!e) return;
  if (!e->plan_only) {
    if (e->stream) (void)hipStreamSynchronize(e->stream);
    for (hipStream_t x : e->xs)
      if (x) (void)hipStreamSynchronize(x);
    for (int i = 0; i < kStageSlots; ++i) {
      if (e->stage[i].buf) (void)hipHostFree(e->stage[i].buf);
      if (e->ev[i]) (void)hipEventDestroy(e->ev[i]);
    }
    if (e->pinned_out) (void)hipHostFree(e->pinned_out);
    for (auto& t : e->timed) { (void)hipEventDestroy(t.a); (void)hipEventDestroy(t.b); }
    for (hipEvent_t v : e->ev_pool) (void)hipEventDestroy(v);
    if (e->copy_stream) (void)hipStreamDestroy(e->copy_stream);
    for (hipStream_t x : e->xs)
      if (x) (void)hipStreamDestroy(x);
    for (hipEvent_t v : e->ev_join)
      if (v) (void)hipEventDestroy(v);
    if (e->ev_fork) (void)hipEventDestroy(e->ev_fork);
  }
  delete e;
}

moa_status moa_load_expert(moa_engine* e, const moa_model_cfg* mc, const void* host_weights, size_t nbytes,
                           int32_t* model_id) {
  if (!e || !mc || !host_weights || !model_id) return MOA_EINVAL;
  if (e->broken) return MOA_ESTATE;
  if (e->step_idx > 0) return MOA_ESTATE;
  const moa_model_cfg& g = e->cfg.model;
  if (mc->n_layers != g.n_layers || mc->d_model != g.d_model || mc->n_heads != g.n_heads ||
      mc->n_kv_heads != g.n_kv_heads || mc->head_dim != g.head_dim || mc->ffn_dim != g.ffn_dim ||
      mc->vocab != g.vocab || mc->rope_theta != g.rope_theta || mc->rms_eps != g.rms_eps)
    return MOA_EINVAL;
  const size_t esz = e->lay.esz;
  const int64_t d = g.d_model, hd = g.head_dim, nh = g.n_heads, nkv = g.n_kv_heads, V = g.vocab, F = g.ffn_dim,
                Lr = g.n_layers;
  const int64_t qd = nh * hd, kd = nkv * hd, qkv = qd + 2 * kd;
  const size_t expect = (size_t)(2 * V * d + d + Lr * (2 * d + qkv * d + d * qd + 3 * F * d)) * esz;
  if (nbytes != expect) return MOA_EINVAL;
  if ((int)e->models.size() >= e->cfg.max_models) return MOA_ENOMEM;

  ModelDev M;
  if (e->plan_only) {
    *model_id = (int32_t)e->models.size();
    e->models.push_back(M);
    return MOA_OK;
  }
  const char* src = (const char*)host_weights;
  size_t so = 0;
  auto next = [&](int64_t n) { const char* p = src + so; so += (size_t)n * esz; return p; };
  size_t mo = e->model_top;
  const size_t mend = mo + e->lay.model_bytes;
  auto dev_take = [&](int64_t n) -> char* {
    char* p = e->arena + mo;
    mo = align_up(mo + (size_t)n * esz, 256);
    return p;
  };
  std::vector<char> tmp;
  auto put_raw = [&](const char* s, int64_t n) -> const void* {
    char* p = dev_take(n);
    if (hipMemcpy(p, s, (size_t)n * esz, hipMemcpyHostToDevice) != hipSuccess) return nullptr;
    return p;
  };
  // matrix built from row sources (bf16: tile-shuffled; f32: row-major)
  auto put_mat = [&](int64_t N, int64_t K, auto rowfn) -> const void* {
    char* p = dev_take(N * K);
    tmp.resize((size_t)N * K * esz);
    if (e->bf16) {
      shuffle_bf16((uint16_t*)tmp.data(), N, K, [&](int64_t n) { return (const uint16_t*)rowfn(n); });
    } else {
      for (int64_t n = 0; n < N; ++n) std::memcpy(tmp.data() + (size_t)n * K * esz, rowfn(n), (size_t)K * esz);
    }
    if (hipMemcpy(p, tmp.data(), tmp.size(), hipMemcpyHostToDevice) != hipSuccess) return nullptr;
    return p;
  };
  bool ok = true;
  auto chk = [&](const void* p) { if (!p) ok = false; return p; };
  M.embed = chk(put_raw(next(V * d), V * d));
  for (int64_t l = 0; l < Lr && ok; ++l) {
    const char* an = next(d);
    const char* wq = next(qd * d);
    const char* wk = next(kd * d);
    const char* wv = next(kd * d);
    const char* wo = next(d * qd);
    const char* mn = next(d);
    const char* wg = next(F * d);
    const char* wu = next(F * d);
    const char* wd = next(d * F);
    M.attn_norm.push_back(chk(put_raw(an, d)));
    M.wqkv.push_back(chk(put_mat(qkv, d, [&](int64_t n) {
      if (n < qd) return wq + (size_t)n * d * esz;
      if (n < qd + kd) return wk + (size_t)(n - qd) * d * esz;
      return wv + (size_t)(n - qd - kd) * d * esz;
    })));
    M.wo.push_back(chk(put_mat(d, qd, [&](int64_t n) { return wo + (size_t)n * qd * esz; })));
    M.mlp_norm.push_back(chk(put_raw(mn, d)));
    if (e->bf16) {
      // 16-row tiles alternate gate / up so a wavefront owning tiles (2i, 2i+1)
      // holds gate and up of the same hidden units.
      M.wgu.push_back(chk(put_mat(2 * F, d, [&](int64_t n) {
        const int64_t t = n / 16, r = n % 16, unit = (t / 2) * 16 + r;
        return ((t & 1) ? wu : wg) + (size_t)unit * d * esz;
      })));
    } else {
      M.wgu.push_back(chk(put_mat(2 * F, d, [&](int64_t n) {
        return n < F ? wg + (size_t)n * d * esz : wu + (size_t)(n - F) * d * esz;
      })));
    }
    M.wdown.push_back(chk(put_mat(d, F, [&](int64_t n) { return wd + (size_t)n * F * esz; })));
  }
  if (ok) M.final_norm = chk(put_raw(next(d), d));
  if (ok) {
    const char* lm = next(V * d);
    M.lm_head = chk(put_mat(V, d, [&](int64_t n) { return lm + (size_t)n * d * esz; }));
  }
  if (!ok) return hip_fail(e, hipErrorUnknown, "moa_load_expert copy");
  if (mo > mend || mo > e->arena_bytes) return hip_fail(e, hipErrorOutOfMemory, "moa_load_expert layout");
  e->model_top = e->lay.off_models + e->lay.model_bytes * (e->models.size() + 1);
  *model_id = (int32_t)e->models.size();
  e->models.push_back(std::move(M));
  return MOA_OK;
}

moa_status moa_submit(moa_engine* e, const int32_t* tokens, int32_t n_tokens, int32_t model_id,
                      int32_t max_new_tokens, int64_t* request_id) {
  if (!e || !request_id) return MOA_EINVAL;
  if (e->broken) return MOA_ESTATE;
  if (!tokens || n_tokens < 1 || max_new_tokens < 1) return MOA_EINVAL;
  if (model_id < 0 || model_id >= (int32_t)e->models.size()) return MOA_EINVAL;
  if ((int64_t)n_tokens + max_new_tokens - 1 > e->cfg.max_model_len) return MOA_EINVAL;
  if (e->cfg.max_prefill_tokens < 1) return MOA_EINVAL;     // a prompt could never be processed
  if (!e->plan_only)   // a dry run never reads token values (its collected tokens are -1)
    for (int32_t i = 0; i < n_tokens; ++i)
      if (tokens[i] < 0 || tokens[i] >= e->cfg.model.vocab) return MOA_EINVAL;
  const int64_t need = ((int64_t)n_tokens + max_new_tokens - 1 + kBlock - 1) / kBlock;
  if (need > e->cfg.num_kv_blocks) return MOA_ENOSPC;
  if (e->live == 0) e->tok_top = 0, e->bt_top = 0;    // stores are empty again: restart them
  if (e->tok_top + n_tokens + max_new_tokens > e->lay.token_store) return MOA_ENOMEM;
  Request r;
  r.id = (int64_t)e->reqs.size();
  r.model = model_id;
  r.P = n_tokens;
  r.G = max_new_tokens;
  r.need = (int32_t)need;
  r.tok_off = e->tok_top;
  e->tok_top += (int64_t)n_tokens + max_new_tokens;
  r.prompt.assign(tokens, tokens + n_tokens);
  e->reqs.push_back(std::move(r));
  e->pending.push_back(e->reqs.back().id);
  e->live += 1;
  *request_id = e->reqs.back().id;
  return MOA_OK;
}

moa_status moa_submit_with_history(moa_engine* e, int32_t model_id, int32_t seed_token, int32_t ctx_len,
                                   const void* host_kv, int32_t max_new_tokens, int64_t* request_id) {
  if (!e || !request_id) return MOA_EINVAL;
  if (e->broken) return MOA_ESTATE;
  if (ctx_len < 0 || max_new_tokens < 1) return MOA_EINVAL;
  if (model_id < 0 || model_id >= (int32_t)e->models.size()) return MOA_EINVAL;
  if ((int64_t)ctx_len + max_new_tokens > e->cfg.max_model_len) return MOA_EINVAL;
  if (!e->plan_only && (seed_token < 0 || seed_token >= e->cfg.model.vocab)) return MOA_EINVAL;
  const int64_t need = ((int64_t)ctx_len + max_new_tokens + kBlock - 1) / kBlock;
  if (need > e->cfg.num_kv_blocks) return MOA_ENOSPC;
  if (e->live == 0) e->tok_top = 0, e->bt_top = 0;
  if (e->tok_top + 1 + max_new_tokens > e->lay.token_store) return MOA_ENOMEM;
  Request r;
  r.id = (int64_t)e->reqs.size();
  r.model = model_id;
  r.shift = ctx_len;
  r.P = ctx_len + 1;
  r.pre = r.P;                        // nothing to prefill
  r.G = max_new_tokens;
  r.need = (int32_t)need;
  r.history = true;
  r.tok_off = e->tok_top;
  e->tok_top += 1 + max_new_tokens;
  r.prompt.assign(1, seed_token);
  if (host_kv && ctx_len > 0 && !e->plan_only) {
    const moa_model_cfg& g = e->cfg.model;
    const size_t bytes = (size_t)g.n_layers * 2 * ctx_len * g.n_kv_heads * g.head_dim * e->lay.esz;
    r.host_kv.assign((const char*)host_kv, (const char*)host_kv + bytes);
  }
  e->reqs.push_back(std::move(r));
  e->pending.push_back(e->reqs.back().id);
  e->live += 1;
  *request_id = e->reqs.back().id;
  return MOA_OK;
}

namespace {

// Write the injected K/V history of admitted requests into their blocks.
// With caller data: stage it through the logits buffer (idle between steps;
// the stream is drained first) one (layer, K|V) position range at a time and
// scatter it with a kernel. Without: fill on the device from a hash of
// (request, layer, K|V, position, head, dim).
moa_status write_histories(moa_engine* e, const std::vector<int64_t>& admitted) {
  const moa_model_cfg& g = e->cfg.model;
  const size_t esz = e->lay.esz;
  const size_t row = (size_t)g.n_kv_heads * g.head_dim;             // elements per position
  const size_t cap_rows = std::max<size_t>(1, (size_t)e->lay.Rmax * g.vocab * 4 / (row * esz));
  bool drained = false;
  for (int64_t id : admitted) {
    Request& r = e->reqs[id];
    if (!r.history || r.shift == 0) continue;
    if (r.host_kv.empty()) {
      HIPCHK(launch_kv_fill(e->stream, e->bf16, e->kv, e->bt_store + r.bt_off, r.shift, g.n_layers,
                            e->cfg.num_kv_blocks, g.n_kv_heads, g.head_dim, (uint32_t)r.id), "history fill");
      continue;
    }
    if (!drained) {
      HIPCHK(hipStreamSynchronize(e->stream), "history sync");
      drained = true;
    }
    for (int l = 0; l < g.n_layers; ++l)
      for (int kv = 0; kv < 2; ++kv)
        for (size_t p0 = 0; p0 < (size_t)r.shift; p0 += cap_rows) {
          const size_t n = std::min(cap_rows, (size_t)r.shift - p0);
          const char* src = r.host_kv.data() + (((size_t)l * 2 + kv) * r.shift + p0) * row * esz;
          HIPCHK(hipMemcpy(e->logits, src, n * row * esz, hipMemcpyHostToDevice), "history upload");
          HIPCHK(launch_kv_scatter(e->stream, e->bf16, e->logits, e->kv, e->bt_store + r.bt_off, (int)p0, (int)n, l,
                                   kv, e->cfg.num_kv_blocks, g.n_kv_heads, g.head_dim), "history scatter");
          HIPCHK(hipStreamSynchronize(e->stream), "history sync");
        }
    std::vector<char>().swap(r.host_kv);
  }
  return MOA_OK;
}

// Wait until staging slot `slot` is no longer read by an in-flight step.
moa_status wait_slot(moa_engine* e, int slot) {
  if (e->ev_step[slot] >= 0) HIPCHK(hipEventSynchronize(e->ev[slot]), "staging wait");
  return MOA_OK;
}

moa_status ensure_stage(moa_engine* e, int slot, size_t bytes) {
  auto& s = e->stage[slot];
  if (s.cap >= bytes) return MOA_OK;
  if (s.buf) HIPCHK(hipHostFree(s.buf), "hipHostFree");
  s.buf = nullptr;
  s.cap = 0;
  size_t cap = std::max(bytes, (size_t)1 << 20);
  HIPCHK(hipHostMalloc((void**)&s.buf, cap, hipHostMallocDefault), "hipHostMalloc");
  s.cap = cap;
  return MOA_OK;
}

int64_t nslots_total(const moa_engine* e) {
  int64_t n = 0;
  for (const ReduceItem& r : e->red) n += r.nslots;
  return n;
}

// Bytes of the library scratch an allocation-free step of this engine may
// need: split-K partials of every model stream and the split-KV attention
// partials, at their planned capacities (the plan is the same as moa_step's).
size_t noalloc_scratch_bytes(const moa_engine* e) {
  const Layout& L = e->lay;
  const moa_model_cfg& g = e->cfg.model;
  const size_t part = align_up((size_t)L.part_cap * 4, 256);
  const size_t pacc = align_up((size_t)L.slots_cap * g.n_heads * g.head_dim * 4, 256);
  const size_t pml = align_up((size_t)L.slots_cap * g.n_heads * 2 * 4, 256);
  return part * (size_t)e->nstreams + pacc + pml;
}

moa_status enqueue_step(moa_engine* e, const std::vector<int64_t>& admitted, int T, int R,
                        const int* grp_rows, const int* grp_lm, bool noalloc) {
  const moa_model_cfg& g = e->cfg.model;
  const Layout& L = e->lay;
  const int slot = (int)(e->step_idx % kStageSlots);
  moa_status st = wait_slot(e, slot);
  if (st != MOA_OK) return st;
  e->keepalive[slot].clear();                 // the step that read them has completed

  // partial sums: the arena's workspace, or this GPU's library scratch
  float* part = e->part;
  float* xpart[kMaxShares - 1];
  for (int k = 0; k < kMaxShares - 1; ++k) xpart[k] = e->xpart[k];
  float* pacc = e->pacc;
  float* pml = e->pml;
  if (noalloc) {
    char* sc = (char*)e->scratch;
    const size_t pb = align_up((size_t)L.part_cap * 4, 256);
    part = (float*)sc;
    for (int k = 0; k < kMaxShares - 1; ++k) xpart[k] = k + 1 < e->nstreams ? (float*)(sc + pb * (k + 1)) : nullptr;
    pacc = (float*)(sc + pb * e->nstreams);
    pml = (float*)(sc + pb * e->nstreams + align_up((size_t)L.slots_cap * g.n_heads * g.head_dim * 4, 256));
  }

  // ---- stage: metadata, then prompts and block lists of admitted requests
  // (an allocation-free step stages only the metadata, in the slot sized for
  // it at moa_create, and uploads prompts and block lists from host copies)
  const int nitems = (int)e->items.size(), nred = (int)e->red.size(), npre = (int)e->pitems.size();
  size_t meta_ints = 4 * (size_t)T + 2 * (size_t)R + 8 * (size_t)nitems + 4 * (size_t)nred + 4 * (size_t)npre;
  size_t up_ints = 0;
  if (!noalloc)
    for (int64_t id : admitted) up_ints += e->reqs[id].prompt.size() + e->reqs[id].blocks.size();
  if (noalloc && e->stage[slot].cap < meta_ints * 4) return hip_fail(e, hipErrorOutOfMemory, "staging size");
  st = ensure_stage(e, slot, (meta_ints + up_ints) * 4);
  if (st != MOA_OK) return st;
  int* hb = (int*)e->stage[slot].buf;
  size_t o = 0;
  auto put = [&](const void* p, size_t n_int) { std::memcpy(hb + o, p, n_int * 4); o += n_int; };
  const size_t o_tok = o; put(e->r_tok.data(), T);
  const size_t o_pos = o; put(e->r_pos.data(), T);
  const size_t o_bt = o; put(e->r_bt.data(), T);
  const size_t o_mod = o; put(e->r_model.data(), T);
  const size_t o_ls = o; put(e->l_src.data(), R);
  const size_t o_ld = o; put(e->l_dst.data(), R);
  const size_t o_it = o; put(e->items.data(), 8 * (size_t)nitems);
  const size_t o_rd = o; put(e->red.data(), 4 * (size_t)nred);
  const size_t o_pi = o; put(e->pitems.data(), 4 * (size_t)npre);
  HIPCHK(hipMemcpyAsync(e->meta, hb, meta_ints * 4, hipMemcpyHostToDevice, e->stream), "meta upload");
  for (int64_t id : admitted) {
    Request& r = e->reqs[id];
    if (noalloc) {
      // r.blocks lives as long as the request; the prompt copy until this step completes
      HIPCHK(hipMemcpyAsync(e->tok_store + r.tok_off, r.prompt.data(), r.prompt.size() * 4, hipMemcpyHostToDevice,
                            e->stream), "prompt upload");
      HIPCHK(hipMemcpyAsync(e->bt_store + r.bt_off, r.blocks.data(), r.blocks.size() * 4, hipMemcpyHostToDevice,
                            e->stream), "block list upload");
      e->keepalive[slot].push_back(std::move(r.prompt));
      r.prompt = std::vector<int32_t>();
      continue;
    }
    const size_t a = o;
    put(r.prompt.data(), r.prompt.size());
    HIPCHK(hipMemcpyAsync(e->tok_store + r.tok_off, hb + a, r.prompt.size() * 4, hipMemcpyHostToDevice, e->stream),
           "prompt upload");
    const size_t b = o;
    put(r.blocks.data(), r.blocks.size());
    HIPCHK(hipMemcpyAsync(e->bt_store + r.bt_off, hb + b, r.blocks.size() * 4, hipMemcpyHostToDevice, e->stream),
           "block list upload");
    std::vector<int32_t>().swap(r.prompt);
  }
  st = write_histories(e, admitted);
  if (st != MOA_OK) return st;
  StepDev sd;
  sd.row_tok = e->meta + o_tok;
  sd.row_pos = e->meta + o_pos;
  sd.row_bt = e->meta + o_bt;
  sd.row_model = e->meta + o_mod;
  sd.lm_src = e->meta + o_ls;
  sd.lm_dst = e->meta + o_ld;
  sd.items = (const AttnItem*)(e->meta + o_it);
  sd.red = (const ReduceItem*)(e->meta + o_rd);
  sd.pre = (const PrefillItem*)(e->meta + o_pi);

  // ---- kernels
  const bool bf = e->bf16;
  const int M = (int)e->models.size();
  const int d = g.d_model, hd = g.head_dim, nh = g.n_heads, nkv = g.n_kv_heads, F = g.ffn_dim, V = g.vocab;
  const int qkv = (nh + 2 * nkv) * hd;
  const size_t xn_lo = (size_t)L.Tmax * d, ao_lo = (size_t)L.Tmax * nh * hd, h_lo = (size_t)L.Tmax * F;
  hipStream_t s = e->stream;
  ModelPtrs mp{};
  auto fill = [&](auto get) { for (int m = 0; m < M; ++m) mp.p[m] = get(e->models[m]); return mp; };

  // one group per model with rows, in the step's row order
  GemmPlanIn gin;
  int gmodel[kMaxModels];
  int r0 = 0;
  for (int i = 0; i < M; ++i) {
    const int m = e->morder[i];
    if (grp_rows[m] == 0) continue;
    gin.row0[gin.ngroups] = r0;
    gin.nrows[gin.ngroups] = grp_rows[m];
    gin.W[gin.ngroups] = nullptr;
    gmodel[gin.ngroups] = m;
    r0 += grp_rows[m];
    gin.ngroups++;
  }
  auto weights = [&](auto get) { GemmPlanIn w = gin; for (int k = 0; k < w.ngroups; ++k) w.W[k] = get(e->models[gmodel[k]]); return w; };

  // kernel timing takes events from a pool that may grow: never in an allocation-free step
  e->time_now = step_is_timed(e, noalloc);
  if (e->time_now && e->timed.size() > 16384) {
    moa_status rs = resolve_timed(e);
    if (rs != MOA_OK) return rs;
  }
  const double esz = (double)L.esz;
  // algorithmic bytes / flops of one grouped GEMM launch
  auto gemm_cost = [&](const GemmArgs& a, int epi, double& bytes, double& flops) {
    double rows = 0;
    for (int k = 0; k < a.ngroups; ++k) rows += a.g[k].nrows;
    const double out_elems = epi == EPI_SWIGLU ? rows * a.N / 2 : rows * a.N;
    bytes = a.ngroups * (double)a.N * a.K * esz + rows * a.K * 4.0 + out_elems * 4.0;
    flops = 2.0 * rows * a.N * a.K;
  };

  // Each stream's share of the layers: rows [r0, r0 + nr), model groups
  // [g0, g0 + ng) and its slices of the item lists. Every buffer the layers
  // touch is indexed by row (or by the row's partial slots and KV blocks),
  // except the split-K partials, which take one buffer per stream.
  struct Share {
    hipStream_t st;
    float* part;
    int r0, nr, g0, ng;
    const AttnItem* items;
    const ReduceItem* red;
    const PrefillItem* pre;
    int nitems, nred, npre, max_item_blocks, pre_max_keys;
    double attn_bytes, attn_flops, pre_bytes, pre_flops, red_bytes;
    int prev_split;
    size_t prev_stride;
  };
  const int nshare = e->nshare;
  Share sh[kMaxShares];
  for (int u = 0; u < nshare; ++u) {
    Share& b = sh[u];
    b.st = u == 0 ? e->stream : e->xs[u - 1];
    b.part = u == 0 ? part : xpart[u - 1];
    b.r0 = e->sh_row[u];
    b.nr = e->sh_row[u + 1] - e->sh_row[u];
    b.g0 = e->sh_group[u];
    b.ng = e->sh_group[u + 1] - e->sh_group[u];
    const int i0 = e->sh_item[u], d0 = e->sh_red[u], p0 = e->sh_pre[u];
    b.nitems = e->sh_item[u + 1] - i0;
    b.nred = e->sh_red[u + 1] - d0;
    b.npre = e->sh_pre[u + 1] - p0;
    b.items = sd.items + i0;
    b.red = sd.red + d0;
    b.pre = sd.pre + p0;
    double kv_keys = 0;
    b.max_item_blocks = 1;
    for (int i = i0; i < i0 + b.nitems; ++i) {
      const AttnItem& it = e->items[i];
      kv_keys += it.k1 - it.k0;
      b.max_item_blocks = std::max(b.max_item_blocks, ((it.k1 - 1) >> 4) - (it.k0 >> 4) + 1);
    }
    // causal prefill blocks: K/V of keys [0, pos0 + nq) once per KV head; q.k and p.v per (row, key <= pos)
    double pre_keys = 0, pre_pairs = 0, pre_rows = 0;
    b.pre_max_keys = 1;
    for (int i = p0; i < p0 + b.npre; ++i) {
      const PrefillItem& pi = e->pitems[i];
      pre_keys += pi.pos0 + pi.nq;
      b.pre_max_keys = std::max(b.pre_max_keys, pi.pos0 + pi.nq);
      pre_pairs += (double)pi.nq * pi.pos0 + (double)pi.nq * (pi.nq + 1) / 2;
      pre_rows += pi.nq;
    }
    double nsl = 0;
    for (int i = d0; i < d0 + b.nred; ++i) nsl += e->red[i].nslots;
    b.pre_bytes = pre_keys * nkv * 2.0 * hd * esz + pre_rows * nh * hd * 8.0;
    b.pre_flops = pre_pairs * nh * hd * 4.0;
    b.attn_bytes = kv_keys * nkv * 2.0 * hd * esz + (double)b.nr * nh * hd * 8.0;
    b.attn_flops = kv_keys * nh * hd * 4.0;
    b.red_bytes = nsl * nh * (hd + 2) * 4.0;
    b.prev_split = 0;
    b.prev_stride = 0;
  }
  double gb = 0, gf = 0;

  if (T > 0) {
    if (nshare > 1) HIPCHK(hipEventRecord(e->ev_fork, s), "stream fork");
    for (int u = 1; u < nshare; ++u) HIPCHK(hipStreamWaitEvent(e->xs[u - 1], e->ev_fork, 0), "stream fork");
    for (int u = 0; u < nshare; ++u) {
      const Share& b = sh[u];
      LAUNCH(MOA_K_EMBED, (double)b.nr * d * (4.0 + esz), 0,
             launch_embed(b.st, bf, e->tok_store, sd.row_tok + b.r0, sd.row_model + b.r0,
                          fill([](const ModelDev& x) { return x.embed; }), e->x + (size_t)b.r0 * d, b.nr, d),
             "embed");
    }
    for (int l = 0; l < g.n_layers; ++l) {
      for (int u = 0; u < nshare; ++u) {
        Share& b = sh[u];
        hipStream_t st = b.st;
        const size_t ro = (size_t)b.r0;
        void* xn_b = (char*)e->xn + ro * d * L.esz;
        const double norm_bytes = (double)b.nr * d * 12.0;
        GemmArgs ga;
        int mt, nt;
        bool lg;
        LAUNCH(MOA_K_NORM, norm_bytes + b.prev_split * (double)b.nr * d * 4.0, 0,
               launch_add_rmsnorm(st, bf, e->x + ro * d, b.prev_split ? b.part + ro * d : nullptr, b.prev_split,
                                  b.prev_stride, nullptr, sd.row_model + ro, b.nr,
                                  fill([l](const ModelDev& x) { return x.attn_norm[l]; }), xn_b, xn_lo, d,
                                  g.rms_eps), "attn norm");
        plan_gemm(e, weights([l](const ModelDev& x) { return x.wqkv[l]; }), b.g0, b.ng, d, qkv, EPI_F32, e->xn,
                  xn_lo, b.part, nullptr, 0, true, ga, mt, nt, lg);
        gemm_cost(ga, EPI_F32, gb, gf);
        LAUNCH_GEMM(MOA_K_GEMM_QKV, lg, gb, gf, launch_gemm(st, bf, ga, EPI_F32, mt, nt), "qkv gemm");
        LAUNCH(MOA_K_ROPE_KV, (double)b.nr * qkv * 4.0 * ga.S + (double)b.nr * (nh * hd * 4.0 + 2.0 * nkv * hd * esz), 0,
               launch_rope_kv(st, bf, b.part + ro * qkv, ga.S, ga.out_split, sd.row_pos + ro, sd.row_bt + ro,
                              e->bt_store, e->rope, e->q + ro * nh * hd, e->kv, l, e->cfg.num_kv_blocks, nh, nkv, hd,
                              b.nr), "rope kv");
        if (b.npre > 0)
          LAUNCH(MOA_K_PREFILL_ATTN, b.pre_bytes, b.pre_flops,
                 launch_prefill_attention(st, b.pre, b.npre, b.pre_max_keys, e->q, e->kv, e->bt_store, l,
                                          e->cfg.num_kv_blocks, nh, nkv, hd, 1.0f / std::sqrt((float)hd), e->ao,
                                          ao_lo), "prefill attention");
        if (b.nitems > 0)
          LAUNCH(MOA_K_ATTN, b.attn_bytes, b.attn_flops,
                 launch_attention(st, bf, b.items, b.nitems, b.max_item_blocks, e->q, e->kv, e->bt_store, sd.row_bt,
                                  l, e->cfg.num_kv_blocks, nh, nkv, hd, 1.0f / std::sqrt((float)hd), e->ao, ao_lo,
                                  pacc, pml), "attention");
        if (b.nred > 0)
          LAUNCH(MOA_K_ATTN_REDUCE, b.red_bytes, 0,
                 launch_attn_reduce(st, bf, b.red, b.nred, pacc, pml, e->ao, ao_lo, nh, hd), "attn reduce");
        plan_gemm(e, weights([l](const ModelDev& x) { return x.wo[l]; }), b.g0, b.ng, nh * hd, d, EPI_F32, e->ao,
                  ao_lo, b.part, nullptr, 0, true, ga, mt, nt, lg);
        gemm_cost(ga, EPI_F32, gb, gf);
        LAUNCH_GEMM(MOA_K_GEMM_O, lg, gb, gf, launch_gemm(st, bf, ga, EPI_F32, mt, nt), "o gemm");
        LAUNCH(MOA_K_NORM, norm_bytes + ga.S * (double)b.nr * d * 4.0, 0,
               launch_add_rmsnorm(st, bf, e->x + ro * d, b.part + ro * d, ga.S, ga.out_split, nullptr,
                                  sd.row_model + ro, b.nr, fill([l](const ModelDev& x) { return x.mlp_norm[l]; }),
                                  xn_b, xn_lo, d, g.rms_eps), "mlp norm");
        if (bf) {
          plan_gemm(e, weights([l](const ModelDev& x) { return x.wgu[l]; }), b.g0, b.ng, d, 2 * F, EPI_SWIGLU,
                    e->xn, xn_lo, nullptr, (uint16_t*)e->h, h_lo, false, ga, mt, nt, lg);
          gemm_cost(ga, EPI_SWIGLU, gb, gf);
          LAUNCH_GEMM(MOA_K_GEMM_GATEUP, lg, gb, gf, launch_gemm(st, bf, ga, EPI_SWIGLU, mt, nt), "gate-up gemm");
        } else {
          plan_gemm(e, weights([l](const ModelDev& x) { return x.wgu[l]; }), b.g0, b.ng, d, 2 * F, EPI_F32, e->xn, 0,
                    b.part, nullptr, 0, false, ga, mt, nt, lg);
          gemm_cost(ga, EPI_F32, gb, gf);
          LAUNCH_GEMM(MOA_K_GEMM_GATEUP, lg, gb, gf, launch_gemm(st, bf, ga, EPI_F32, mt, nt), "gate-up gemm");
          HIPCHK(launch_swiglu_f32(st, b.part + ro * 2 * F, (float*)e->h + ro * F, b.nr, F), "swiglu");
        }
        plan_gemm(e, weights([l](const ModelDev& x) { return x.wdown[l]; }), b.g0, b.ng, F, d, EPI_F32, e->h, h_lo,
                  b.part, nullptr, 0, true, ga, mt, nt, lg);
        gemm_cost(ga, EPI_F32, gb, gf);
        LAUNCH_GEMM(MOA_K_GEMM_DOWN, lg, gb, gf, launch_gemm(st, bf, ga, EPI_F32, mt, nt), "down gemm");
        b.prev_split = ga.S;
        b.prev_stride = ga.out_split;
      }
    }
    // Final norm, LM head and argmax of each share's emitting rows, in LM-row
    // order (the LM head's own input rows and the logits rows are disjoint
    // across shares), before the join.
    if (R > 0) {
      const size_t xl_lo = (size_t)L.Rmax * d;
      GemmPlanIn lin;
      int lfirst[kMaxModels + 1];     // LM groups of row groups [0, k): lfirst[k]
      int lr0 = 0;
      for (int k = 0; k < gin.ngroups; ++k) {
        lfirst[k] = lin.ngroups;
        const int m = gmodel[k];
        if (grp_lm[m] == 0) continue;
        lin.row0[lin.ngroups] = lr0;
        lin.nrows[lin.ngroups] = grp_lm[m];
        lin.W[lin.ngroups] = e->models[m].lm_head;
        lr0 += grp_lm[m];
        lin.ngroups++;
      }
      lfirst[gin.ngroups] = lin.ngroups;
      for (int u = 0; u < nshare; ++u) {
        const Share& b = sh[u];
        const int b0 = e->sh_lm[u], nb = e->sh_lm[u + 1] - e->sh_lm[u];
        if (nb == 0) continue;
        const int lg0 = lfirst[b.g0], lng = lfirst[b.g0 + b.ng] - lg0;
        LAUNCH(MOA_K_NORM, (double)nb * d * (12.0 + b.prev_split * 4.0), 0,
               launch_add_rmsnorm(b.st, bf, e->x, b.part, b.prev_split, b.prev_stride, sd.lm_src + b0, sd.row_model,
                                  nb, fill([](const ModelDev& x) { return x.final_norm; }),
                                  (char*)e->xl + (size_t)b0 * d * L.esz, xl_lo, d, g.rms_eps), "final norm");
        GemmArgs ga;
        int mt, nt;
        bool lg;
        plan_gemm(e, lin, lg0, lng, d, V, EPI_F32, e->xl, xl_lo, e->logits, nullptr, 0, false, ga, mt, nt, lg);
        gemm_cost(ga, EPI_F32, gb, gf);
        LAUNCH_GEMM(MOA_K_GEMM_LMHEAD, lg, gb, gf, launch_gemm(b.st, bf, ga, EPI_F32, mt, nt), "lm head");
        LAUNCH(MOA_K_ARGMAX, (double)nb * V * 4.0, 0,
               launch_argmax(b.st, e->logits + (size_t)b0 * V, nb, V, sd.lm_dst + b0, e->tok_store), "argmax");
      }
    }
    for (int u = 1; u < nshare; ++u) {
      HIPCHK(hipEventRecord(e->ev_join[u - 1], e->xs[u - 1]), "stream join");
      HIPCHK(hipStreamWaitEvent(s, e->ev_join[u - 1], 0), "stream join");
    }
  }
  (void)L;
  HIPCHK(hipEventRecord(e->ev[slot], s), "event record");
  e->ev_step[slot] = e->step_idx;
  return MOA_OK;
}

}  // namespace

}  // extern "C"

namespace {

moa_status step_impl(moa_engine* e, moa_step_info* info, bool noalloc) {
  if (info) std::memset(info, 0, sizeof(*info));
  if (e->pending.empty() && e->running.empty()) {
    if (info) { info->step = -1; info->free_blocks = (int32_t)e->free_blocks.nfree; }
    return MOA_OK;
  }
  const int64_t s = e->step_idx;
  const int M = (int)e->models.size();
  // 1 admit
  std::vector<int64_t> admitted;
  while (!e->pending.empty() && (int32_t)e->running.size() < e->cfg.max_num_seqs) {
    Request& r = e->reqs[e->pending.front()];
    if (r.need > e->free_blocks.nfree) break;
    if (e->bt_top + r.need > e->lay.block_store) {        // block-list store full
      if (e->running.empty()) return MOA_ENOMEM;          // nothing will free it before a collect
      break;
    }
    e->free_blocks.take(r.need, r.blocks);
    r.bt_off = e->bt_top;
    e->bt_top += r.need;
    r.admit_step = s;
    r.state = 1;
    e->running.push_back(r.id);
    admitted.push_back(r.id);
    e->pending.pop_front();
  }
  // 2 prefill, 3 decode: record per-request actions in admission order
  struct Act { int64_t id; int kind; int start, len; };   // kind 0 prefill chunk, 1 decode
  std::vector<Act> acts;
  acts.reserve(e->running.size() + 8);
  int budget = e->cfg.max_prefill_tokens;
  int n_pre = 0, n_dec = 0;
  for (int64_t id : e->running) {
    if (budget <= 0) break;
    Request& r = e->reqs[id];
    if (r.pre < r.P) {
      const int c = std::min(r.P - r.pre, budget);
      acts.push_back({id, 0, r.pre, c});
      r.chunks.push_back({s, r.pre, c});
      r.pre += c;
      budget -= c;
      n_pre += c;
      if (r.pre == r.P) { r.gen = 1; r.fresh = true; }
    }
  }
  for (int64_t id : e->running) {
    Request& r = e->reqs[id];
    if (r.pre == r.P && !r.fresh && r.gen < r.G) {
      acts.push_back({id, 1, r.P + r.gen - 1, 1});
      r.gen += 1;
      n_dec += 1;
    }
  }
  // Model order of the step's rows. With several model streams the active
  // models are dealt into one set per stream, largest device cost first to
  // the cheapest set so far (cost: the model's weights, streamed once, plus
  // the K/V bytes its rows' attention reads), and the rows are laid out set
  // by set, so each stream's share is one contiguous run.
  int set_size[kMaxShares] = {0};
  int nsets = 1;
  const int step_streams = step_is_timed(e, noalloc) ? 1 : e->nstreams;
  {
    double cost[kMaxModels] = {0};
    bool active[kMaxModels] = {false};
    const double kv_pos = (double)e->lay.block_bytes / kBlock;   // K/V bytes of one position, all layers
    for (const Act& a : acts) {
      const int m = e->reqs[a.id].model;
      active[m] = true;
      cost[m] += kv_pos * ((double)a.len * a.start + (double)a.len * (a.len + 1) / 2);
    }
    // a model's GEMMs take the longer of streaming its weights and their
    // matrix-core issue, which catches up at ~96 rows (split-bf16 on the
    // 16x16 MFMA against the measured read rate)
    int nrow[kMaxModels] = {0};
    for (const Act& a : acts) nrow[e->reqs[a.id].model] += a.len;
    int am[kMaxModels], na = 0, k = 0;
    for (int m = 0; m < M; ++m)
      if (active[m]) {
        cost[m] += (double)e->lay.model_bytes * std::max(1.0, nrow[m] / 96.0);
        am[na++] = m;
      }
    for (int m = 0; m < M; ++m) e->mcost[m] = cost[m];
    e->nactive = na;
    nsets = std::max(1, std::min(step_streams, na));
    if (nsets > 1) {
      int by_cost[kMaxModels];
      for (int i = 0; i < na; ++i) by_cost[i] = am[i];
      std::stable_sort(by_cost, by_cost + na, [&cost](int a, int b) { return cost[a] > cost[b]; });
      int set_of[kMaxModels];
      double load[kMaxShares] = {0};
      for (int i = 0; i < na; ++i) {
        int best = 0;
        for (int u = 1; u < nsets; ++u)
          if (load[u] < load[best]) best = u;
        load[best] += cost[by_cost[i]];
        set_of[by_cost[i]] = best;
      }
      for (int u = 0; u < nsets; ++u)
        for (int i = 0; i < na; ++i)
          if (set_of[am[i]] == u) { e->morder[k++] = am[i]; set_size[u]++; }
    } else {
      for (int i = 0; i < na; ++i) e->morder[k++] = am[i];
      set_size[0] = na;
    }
    for (int m = 0; m < M; ++m)
      if (!active[m]) e->morder[k++] = m;
  }
  // rows grouped by model in that order: prefill chunks then decode rows, each in admission order
  const int T = n_pre + n_dec;
  e->r_tok.clear(); e->r_pos.clear(); e->r_bt.clear(); e->r_model.clear();
  e->l_src.clear(); e->l_dst.clear(); e->items.clear(); e->red.clear(); e->pitems.clear();
  // bf16 engines run prompt chunks through the causal MFMA prefill kernel
  const bool tiled_prefill = e->bf16 && (e->cfg.model.head_dim == 64 || e->cfg.model.head_dim == 128);
  int grp_rows[kMaxModels] = {0}, grp_lm[kMaxModels] = {0};
  int nslots = 0;
  std::vector<std::pair<int64_t, int>> capture_rows;   // (request, lm row)
  for (int mi = 0; mi < M; ++mi) {
    const int m = e->morder[mi];
    for (int pass = 0; pass < 2; ++pass) {
      for (const Act& a : acts) {
        if (a.kind != pass) continue;
        Request& r = e->reqs[a.id];
        if (r.model != m) continue;
        for (int i = 0; i < a.len; ++i) {
          const int pos = a.start + i;
          const int row = (int)e->r_tok.size();
          e->r_tok.push_back((int)(r.tok_off + pos - r.shift));   // prompt slot, or output gen-1 for decode
          e->r_pos.push_back(pos);
          e->r_bt.push_back((int)r.bt_off);
          e->r_model.push_back(m);
          grp_rows[m]++;
          const int ctx = pos + 1;
          const int bto = (int)r.bt_off;
          if (a.kind == 0 && tiled_prefill) {
            if (i % kPrefillRows == 0) e->pitems.push_back({row, pos, std::min(kPrefillRows, a.len - i), bto});
          } else if (a.kind == 0) {
            e->items.push_back({row, 0, ctx, -1, bto, 0, 0, 0});
          } else {
            const int ns = (ctx + kSplitKeys - 1) / kSplitKeys;
            if (ns == 1) {
              e->items.push_back({row, 0, ctx, -1, bto, 0, 0, 0});
            } else {
              e->red.push_back({row, nslots, ns, 0});
              for (int k = 0; k < ns; ++k)
                e->items.push_back({row, k * kSplitKeys, std::min(ctx, (k + 1) * kSplitKeys), nslots + k,
                                    bto + k * kSplitKeys / kBlock, 0, 0, 0});
              nslots += ns;
            }
          }
          const bool emits = (a.kind == 1) || (pos == r.P - 1);
          if (emits) {
            const int gen_idx = (a.kind == 1) ? (pos - r.P + 1) : 0;   // output index produced
            e->l_src.push_back(row);
            e->l_dst.push_back((int)(r.tok_off + r.P - r.shift + gen_idx));
            grp_lm[m]++;
            if (r.capture) capture_rows.push_back({a.id, (int)e->l_src.size() - 1});
          }
        }
      }
    }
  }
  const int R = (int)e->l_src.size();
  // Shares: the step's model groups dealt out in contiguous runs, one per
  // model stream (rows, LM rows and items follow their groups).
  int ngrp = 0;
  for (int m = 0; m < M; ++m) ngrp += grp_rows[m] > 0;
  const int nshare = std::max(1, std::min(step_streams, ngrp));
  e->nshare = nshare;
  e->sh_group[0] = 0;
  for (int u = 0; u < nshare; ++u) e->sh_group[u + 1] = e->sh_group[u] + set_size[u];
  {
    int u = 0, k = 0, rows = 0, lms = 0;
    e->sh_row[0] = 0;
    e->sh_lm[0] = 0;
    for (int mi = 0; mi < M && u < nshare; ++mi) {
      const int m = e->morder[mi];
      if (!grp_rows[m]) continue;
      rows += grp_rows[m];
      lms += grp_lm[m];
      ++k;
      if (k == e->sh_group[u + 1]) { ++u; e->sh_row[u] = rows; e->sh_lm[u] = lms; }
    }
    e->sh_row[nshare] = T;
    e->sh_lm[nshare] = R;
  }
  const int* shr = e->sh_row;
  auto share_of = [shr, nshare](int row) { int u = 0; while (u + 1 < nshare && row >= shr[u + 1]) ++u; return u; };
  // Launch order of the decode-attention items, per stream: full-length key
  // ranges first, then the shorter ones by decreasing length, so the grid
  // ends on its shortest workgroups. Every item writes its own partial slot
  // (or its row's output), so the order changes no result.
  std::stable_sort(e->items.begin(), e->items.end(), [&share_of](const AttnItem& a, const AttnItem& b) {
    const int sa = share_of(a.row), sb = share_of(b.row);
    if (sa != sb) return sa < sb;
    return a.k1 - a.k0 > b.k1 - b.k0;
  });
  // the split combine in the same spirit: rows with the most partial slots first
  std::stable_sort(e->red.begin(), e->red.end(), [&share_of](const ReduceItem& a, const ReduceItem& b) {
    const int sa = share_of(a.row), sb = share_of(b.row);
    if (sa != sb) return sa < sb;
    return a.nslots > b.nslots;
  });
  // share boundaries in the item lists (prefill items are pushed in row order)
  for (int u = 0; u <= nshare; ++u) e->sh_item[u] = e->sh_red[u] = e->sh_pre[u] = 0;
  for (const AttnItem& it : e->items) e->sh_item[share_of(it.row) + 1]++;
  for (const ReduceItem& rd : e->red) e->sh_red[share_of(rd.row) + 1]++;
  for (const PrefillItem& pi : e->pitems) e->sh_pre[share_of(pi.row0) + 1]++;
  for (int u = 0; u < nshare; ++u) {
    e->sh_item[u + 1] += e->sh_item[u];
    e->sh_red[u + 1] += e->sh_red[u];
    e->sh_pre[u + 1] += e->sh_pre[u];
  }
  if (!e->plan_only) {
    if (T > e->lay.Tmax || R > e->lay.Rmax || nslots > e->lay.slots_cap ||
        (int64_t)e->items.size() > e->lay.items_cap) {
      e->broken = true;
      std::fprintf(stderr, "moa: step plan exceeds workspace (T=%d R=%d slots=%d)\n", T, R, nslots);
      return MOA_EHIP;
    }
    moa_status st = enqueue_step(e, admitted, T, R, grp_rows, grp_lm, noalloc);
    if (st != MOA_OK) return st;
    for (auto& cr : capture_rows) {
      Request& r = e->reqs[cr.first];
      const int row = cr.second;
      const int gen_idx = e->l_dst[row] - (int)(r.tok_off + r.P - r.shift);
      hipError_t err = hipMemcpyAsync(r.capture + (size_t)gen_idx * e->cfg.model.vocab,
                                      e->logits + (size_t)row * e->cfg.model.vocab,
                                      (size_t)e->cfg.model.vocab * 4, hipMemcpyDeviceToHost, e->stream);
      if (err != hipSuccess) return hip_fail(e, err, "logit capture");
    }
  } else {
    for (int64_t id : admitted) std::vector<int32_t>().swap(e->reqs[id].prompt);
  }
  for (int64_t id : admitted) std::vector<char>().swap(e->reqs[id].host_kv);
  // 4 retire
  int n_ret = 0;
  std::vector<int64_t> keep;
  keep.reserve(e->running.size());
  for (int64_t id : e->running) {
    Request& r = e->reqs[id];
    if (r.gen == r.G) {
      e->free_blocks.give(r.blocks);
      r.finish_step = s;
      r.state = 2;
      e->done.push_back(id);
      n_ret++;
    } else {
      keep.push_back(id);
    }
    r.fresh = false;
  }
  e->running.swap(keep);
  e->trace.push_back({s, (int64_t)admitted.size(), n_pre, n_dec, n_ret, e->free_blocks.nfree});
  e->step_idx++;
  if (info) {
    info->step = s;
    info->admitted = (int32_t)admitted.size();
    info->prefill_tokens = n_pre;
    info->decode_rows = n_dec;
    info->finished = n_ret;
    info->running = (int32_t)e->running.size();
    info->pending = (int32_t)e->pending.size();
    info->free_blocks = (int32_t)e->free_blocks.nfree;
    info->emitted = R;
  }
  return MOA_OK;
}

}  // namespace

extern "C" {

moa_status moa_step(moa_engine* e, moa_step_info* info) {
  if (!e) return MOA_EINVAL;
  if (e->broken) return MOA_ESTATE;
  return step_impl(e, info, false);
}

moa_status moa_step_noalloc(moa_engine* e, moa_step_info* info) {
  if (!e) return MOA_EINVAL;
  if (e->broken) return MOA_ESTATE;
  if (noalloc_scratch_bytes(e) > kScratchBytes) {
    if (info) std::memset(info, 0, sizeof(*info));
    return MOA_ENOMEM;
  }
  return step_impl(e, info, true);
}

moa_status moa_collect(moa_engine* e, int64_t upto_step, moa_result* res, int32_t cap, int32_t* n_out,
                       int32_t* tok_buf, int64_t tok_cap) {
  if (!e || !n_out) return MOA_EINVAL;
  if (e->broken) return MOA_ESTATE;
  if (upto_step < 0) upto_step = e->step_idx - 1;
  int32_t n = 0;
  int64_t ntok = 0, last = -1;
  for (int64_t id : e->done) {
    const Request& r = e->reqs[id];
    if (r.finish_step > upto_step) break;          // done is ordered by finish step
    n++;
    ntok += r.G;
    last = std::max(last, r.finish_step);
  }
  *n_out = n;
  if (n == 0) return MOA_OK;
  if (!res || !tok_buf || n > cap || ntok > tok_cap) return MOA_EINVAL;
  if (!e->plan_only) {
    // Wait for the last step that retired one of them (if its staging slot has
    // been reused since, that step already completed), then copy on the side stream.
    for (int i = 0; i < kStageSlots; ++i)
      if (e->ev_step[i] == last) HIPCHK(hipEventSynchronize(e->ev[i]), "collect wait");
    if ((size_t)ntok > e->pinned_out_cap) {
      if (e->pinned_out) HIPCHK(hipHostFree(e->pinned_out), "hipHostFree");
      e->pinned_out = nullptr;
      size_t cap2 = std::max((size_t)ntok, (size_t)1 << 16);
      HIPCHK(hipHostMalloc((void**)&e->pinned_out, cap2 * 4, hipHostMallocDefault), "hipHostMalloc");
      e->pinned_out_cap = cap2;
    }
    int64_t o = 0;
    for (int32_t i = 0; i < n; ++i) {
      const Request& r = e->reqs[e->done[i]];
      HIPCHK(hipMemcpyAsync(e->pinned_out + o, e->tok_store + r.tok_off + r.P - r.shift, (size_t)r.G * 4,
                            hipMemcpyDeviceToHost, e->copy_stream), "collect copy");
      o += r.G;
    }
    HIPCHK(hipStreamSynchronize(e->copy_stream), "collect sync");
    std::memcpy(tok_buf, e->pinned_out, (size_t)ntok * 4);
  } else {
    for (int64_t i = 0; i < ntok; ++i) tok_buf[i] = -1;
  }
  int64_t o = 0;
  for (int32_t i = 0; i < n; ++i) {
    Request& r = e->reqs[e->done[i]];
    res[i].request_id = r.id;
    res[i].model_id = r.model;
    res[i].n_tokens = r.G;
    res[i].tok_offset = o;
    res[i].finish_step = r.finish_step;
    o += r.G;
    r.state = 3;
    r.capture = nullptr;
    e->live -= 1;
  }
  e->done.erase(e->done.begin(), e->done.begin() + n);
  return MOA_OK;
}

moa_status moa_sync(moa_engine* e) {
  if (!e) return MOA_EINVAL;
  if (e->broken) return MOA_ESTATE;
  if (!e->plan_only) HIPCHK(hipStreamSynchronize(e->stream), "sync");
  return MOA_OK;
}

moa_status moa_debug_request(moa_engine* e, int64_t id, moa_request_info* info) {
  if (!e || !info || id < 0 || id >= (int64_t)e->reqs.size()) return MOA_EINVAL;
  const Request& r = e->reqs[id];
  info->model_id = r.model;
  info->prompt_len = r.P;
  info->max_new_tokens = r.G;
  info->n_blocks = (int32_t)r.blocks.size();
  info->admit_step = r.admit_step;
  info->finish_step = r.finish_step;
  info->n_chunks = (int32_t)r.chunks.size();
  info->state = r.state;
  return MOA_OK;
}

moa_status moa_debug_block_table(moa_engine* e, int64_t id, int32_t* out, int32_t cap, int32_t* n_out) {
  if (!e || !n_out || id < 0 || id >= (int64_t)e->reqs.size()) return MOA_EINVAL;
  const Request& r = e->reqs[id];
  *n_out = (int32_t)r.blocks.size();
  if ((int32_t)r.blocks.size() > cap || (!out && !r.blocks.empty())) return MOA_EINVAL;
  if (!r.blocks.empty()) std::memcpy(out, r.blocks.data(), r.blocks.size() * 4);
  return MOA_OK;
}

moa_status moa_debug_chunks(moa_engine* e, int64_t id, int64_t* out, int32_t cap, int32_t* n_out) {
  if (!e || !n_out || id < 0 || id >= (int64_t)e->reqs.size()) return MOA_EINVAL;
  const Request& r = e->reqs[id];
  *n_out = (int32_t)r.chunks.size();
  if ((int32_t)r.chunks.size() > cap || (!out && !r.chunks.empty())) return MOA_EINVAL;
  for (size_t i = 0; i < r.chunks.size(); ++i)
    for (int k = 0; k < 3; ++k) out[3 * i + k] = r.chunks[i][k];
  return MOA_OK;
}

moa_status moa_debug_steps(moa_engine* e, int64_t* out, int64_t cap, int64_t* n_out) {
  if (!e || !n_out) return MOA_EINVAL;
  *n_out = (int64_t)e->trace.size();
  if ((int64_t)e->trace.size() > cap || (!out && !e->trace.empty())) return MOA_EINVAL;
  for (size_t i = 0; i < e->trace.size(); ++i)
    for (int k = 0; k < 6; ++k) out[6 * i + k] = e->trace[i][k];
  return MOA_OK;
}

moa_status moa_debug_time_kernels(moa_engine* e, int32_t every, double peak_bw, double peak_flops) {
  if (!e || !(peak_bw > 0) || !(peak_flops > 0)) return MOA_EINVAL;
  if (e->broken) return MOA_ESTATE;
  if (!e->plan_only) {
    moa_status st = resolve_timed(e);
    if (st != MOA_OK) return st;
  }
  e->time_every = e->plan_only ? 0 : std::max(0, every);
  e->account = true;
  e->peak_bw = peak_bw;
  e->peak_flops = peak_flops;
  for (auto& k : e->kstats) k = moa_kernel_stats{};
  return MOA_OK;
}

moa_status moa_debug_kernel_stats(moa_engine* e, moa_kernel_stats* out) {
  if (!e || !out) return MOA_EINVAL;
  if (e->broken) return MOA_ESTATE;
  if (!e->plan_only) {
    moa_status st = resolve_timed(e);
    if (st != MOA_OK) return st;
  }
  for (int i = 0; i < MOA_K_COUNT; ++i) out[i] = e->kstats[i];
  return MOA_OK;
}

moa_status moa_debug_step_shares(moa_engine* e, int32_t* n_shares, int32_t* n_models, int32_t* models,
                                 double* cost, int32_t* share_models0, int32_t* share_row0,
                                 int32_t* share_lm0) {
  if (!e || !n_shares || !n_models || !models || !cost || !share_models0 || !share_row0 || !share_lm0)
    return MOA_EINVAL;
  *n_shares = e->nshare;
  *n_models = e->nactive;
  for (int i = 0; i < e->nactive; ++i) {
    models[i] = e->morder[i];
    cost[i] = e->mcost[e->morder[i]];
  }
  for (int u = 0; u <= e->nshare; ++u) {
    share_models0[u] = e->sh_group[u];
    share_row0[u] = e->sh_row[u];
    share_lm0[u] = e->sh_lm[u];
  }
  return MOA_OK;
}

moa_status moa_debug_measure_peaks(moa_engine* e, double* read_bytes_per_s, double* mfma_flops_per_s) {
  if (!e || !read_bytes_per_s || !mfma_flops_per_s) return MOA_EINVAL;
  if (e->broken || e->plan_only) return MOA_ESTATE;
  const size_t bytes = std::min(e->lay.kv_bytes, (size_t)8 << 30) & ~(size_t)15;
  if (bytes < ((size_t)1 << 30)) return MOA_EINVAL;
  const size_t sink_bytes = (size_t)e->lay.Rmax * e->cfg.model.vocab * 4;
  const int read_grid = 4096, mfma_grid = 1024, iters = 8192;   // ~2 ms per MFMA run
  if (sink_bytes < (size_t)mfma_grid * 256 * 4 || sink_bytes < (size_t)read_grid * 4) return MOA_EINVAL;
  hipEvent_t a = nullptr, b = nullptr;
  HIPCHK(hipEventCreate(&a), "peaks event");
  HIPCHK(hipEventCreate(&b), "peaks event");
  double best_read = 0, best_mfma = 0;
  for (int rep = 0; rep < 6; ++rep) {
    float ms = 0.f;
    HIPCHK(hipEventRecord(a, e->stream), "peaks event");
    HIPCHK(launch_peak_read(e->stream, e->kv, bytes, (unsigned*)e->logits, read_grid), "peak read");
    HIPCHK(hipEventRecord(b, e->stream), "peaks event");
    HIPCHK(hipEventSynchronize(b), "peaks wait");
    HIPCHK(hipEventElapsedTime(&ms, a, b), "peaks time");
    if (rep > 0 && ms > 0) best_read = std::max(best_read, bytes / (ms * 1e-3));
    HIPCHK(hipEventRecord(a, e->stream), "peaks event");
    HIPCHK(launch_peak_mfma(e->stream, e->logits, mfma_grid, iters), "peak mfma");
    HIPCHK(hipEventRecord(b, e->stream), "peaks event");
    HIPCHK(hipEventSynchronize(b), "peaks wait");
    HIPCHK(hipEventElapsedTime(&ms, a, b), "peaks time");
    if (rep > 0 && ms > 0) best_mfma = std::max(best_mfma, (double)mfma_grid * 4 * iters * 4 * 32768.0 / (ms * 1e-3));
  }
  (void)hipEventDestroy(a);
  (void)hipEventDestroy(b);
  *read_bytes_per_s = best_read;
  *mfma_flops_per_s = best_mfma;
  return MOA_OK;
}

moa_status moa_debug_capture_logits(moa_engine* e, int64_t id, float* host_logits, int64_t cap) {
  if (!e || !host_logits || id < 0 || id >= (int64_t)e->reqs.size()) return MOA_EINVAL;
  Request& r = e->reqs[id];
  if (cap < (int64_t)r.G * e->cfg.model.vocab) return MOA_EINVAL;
  if (r.state >= 2 || (r.pre == r.P && r.gen > 0)) return MOA_ESTATE;
  r.capture = host_logits;
  return MOA_OK;
}

}  // extern "C"
