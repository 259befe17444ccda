// Internal launch interface between the engine's host code and its gfx950
// kernels. Not part of the C ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>
#include <cstddef>

namespace moa {

constexpr int kMaxModels = 8;     // models per engine (grouped launches carry one slot each)
constexpr int kBlock = 16;        // KV slots per block
constexpr int kSplitKeys = 256;   // keys per decode-attention split (fixed: results do not depend on the batch)

struct ModelPtrs { const void* p[kMaxModels]; };

// One contiguous segment of rows that shares a weight matrix.
struct GemmGroup {
  const void* W;    // bf16: tile-shuffled [N/16][K/32][64 lanes][8]; f32: row-major [N][K]
  int row0, nrows;  // rows [row0, row0 + nrows) of X and of the output
  int n_mc;         // row chunks of 16*MT rows
  int item0;        // first wave item of this group
  int mrows;        // medium-M kernel: rows per row chunk (a multiple of 16, at most 16*RT;
                    // 0: 16*RT); the other kernels ignore it
};

constexpr int kMaxGroups = kMaxModels;

struct GemmArgs {
  GemmGroup g[kMaxGroups];
  int ngroups;
  int total_items;
  const void* X;       // [rows][K] activations, row stride K: f32, or the hi plane of a split-bf16 pair
  size_t x_lo;         // bf16: elements from the hi plane to the lo plane (x ~= hi + lo)
  int K, N;
  int S;               // k splits (partial sums out[s])
  int ksteps;          // 32-wide k steps per split
  float* out;          // f32 output / partials: out + s*out_split + row*N + n
  size_t out_split;
  uint16_t* hout;      // SwiGLU epilogue output, split bf16 [rows][N/2] (hi), lo plane at +h_lo
  size_t h_lo;
};

enum Epilogue { EPI_F32 = 0, EPI_SWIGLU = 1 };

// launch_gemm(mt = kWgTile + MT, nt = NT): the workgroup-tile kernel; each item
// is one workgroup of 16*MT rows x 64*NT columns x one k-split (N % (64*NT) == 0).
constexpr int kWgTile = 1000;
// launch_gemm(mt = kMmTile + RT, nt): the medium-M kernel; each item is 16*RT
// rows (RT = 2, 4 or 8) x NW*CT*16 columns x one of S k-splits of K/32/S
// k-steps (rounded; 1 <= S <= K/32), with nt = CT (NW = 4 waves, RT <= 4;
// CT = 2 or 4), nt = 8 + CT (NW = 8 waves; CT = 4 with RT >= 4, CT = 2
// with RT = 8) or nt = 16 + CT (NW = 8 waves, RT = 8, a three-stage weight
// register ring; CT = 2 or 4);
// N must be a multiple of the columns.
constexpr int kMmTile = 3000;

// Attention work item: one query row against keys [k0, k1) of its request.
// bt_off: index in the block store of the block holding key k0 (k0 is a
// multiple of 16). slot < 0: write the final output, else partial slot.
struct AttnItem { int row, k0, k1, slot, bt_off, pad0, pad1, pad2; };
struct ReduceItem { int row, slot0, nslots, pad; };
// Causal prefill block: step rows [row0, row0 + nq) hold positions
// [pos0, pos0 + nq) of one request (nq <= kPrefillRows); keys [0, pos0 + nq).
// bt_off: the request's block list in the block store.
constexpr int kPrefillRows = 128;
struct PrefillItem { int row0, pos0, nq, bt_off; };

struct StepDev {
  const int* row_tok;    // [T] index into the token store
  const int* row_pos;    // [T]
  const int* row_bt;     // [T] offset of the row's block list in the block store
  const int* row_model;  // [T]
  const int* lm_src;     // [R] row that produces a token
  const int* lm_dst;     // [R] token-store slot the token goes to
  const AttnItem* items; // attention items
  const ReduceItem* red; // split-combine items
  const PrefillItem* pre;// causal prefill blocks
};

// Attach a start/stop event pair to the launches that follow (nullptr: none).
void set_launch_events(hipEvent_t start, hipEvent_t stop);

// All launchers enqueue on `st` and return hipGetLastError().
hipError_t launch_embed(hipStream_t st, bool bf16, const int* tok_store, const int* row_tok,
                        const int* row_model, ModelPtrs embed, float* x, int T, int d);

// bf16 mode writes split-bf16 output: hi at out, lo at out + out_lo (elements).
hipError_t launch_add_rmsnorm(hipStream_t st, bool bf16, float* x, const float* part, int nsplit,
                              size_t split_stride, const int* gather, const int* row_model, int nrows,
                              ModelPtrs gamma, void* out, size_t out_lo, int d, float eps);

hipError_t launch_gemm(hipStream_t st, bool bf16, const GemmArgs& a, int epi, int mt, int nt);

hipError_t launch_swiglu_f32(hipStream_t st, const float* gu, float* h, int T, int ffn);

hipError_t launch_rope_kv(hipStream_t st, bool bf16, const float* part, int nsplit, size_t split_stride,
                          const int* row_pos, const int* row_bt, const int* bt_store,
                          const float2* rope_tab, float* q, void* kv, int layer, int num_blocks,
                          int n_h, int n_kv, int hd, int T);

// max_item_blocks: the most KV blocks any item's key range touches (LDS list).
hipError_t launch_attention(hipStream_t st, bool bf16, const AttnItem* items, int nitems, int max_item_blocks,
                            const float* q, const void* kv, const int* bt_store, const int* row_bt,
                            int layer, int num_blocks, int n_h, int n_kv, int hd, float scale,
                            void* out, size_t out_lo, float* pacc, float* pml);

// bf16 KV only, head_dim 64 or 128; writes split-bf16 rows of `out`.
// max_keys: the largest pos0 + nq over the items (their block lists are
// staged in LDS; hipErrorInvalidValue when they do not fit, past ~400k keys).
constexpr unsigned kPrefillLdsMax = 144u * 1024u;
hipError_t launch_prefill_attention(hipStream_t st, const PrefillItem* items, int nitems, int max_keys,
                                   const float* q, const void* kv, const int* bt_store, int layer, int num_blocks,
                                   int n_h, int n_kv, int hd, float scale, void* out, size_t out_lo);

hipError_t launch_attn_reduce(hipStream_t st, bool bf16, const ReduceItem* red, int nred,
                              const float* pacc, const float* pml, void* out, size_t out_lo, int n_h,
                              int hd);

// Injected history. scatter: src [n][n_kv][hd] (engine dtype) -> positions
// [p0, p0 + n) of plane (layer, kv: 0 K / 1 V) through the request's block list.
// fill: positions [0, ctx) of every layer from a hash of (tag, layer, kv,
// position, head, dim), values in [-1, 1).
hipError_t launch_kv_scatter(hipStream_t st, bool bf16, const void* src, void* kv, const int* blocks, int p0, int n,
                             int layer, int kv_sel, int num_blocks, int n_kv, int hd);
hipError_t launch_kv_fill(hipStream_t st, bool bf16, void* kv, const int* blocks, int ctx, int n_layers,
                          int num_blocks, int n_kv, int hd, uint32_t tag);

hipError_t launch_argmax(hipStream_t st, const float* logits, int R, int V, const int* lm_dst,
                         int* tok_store);

// The library's per-GPU scratch array (a file-scope __device__ array of
// kScratchBytes, one copy on every GPU the library runs on, kept until the
// process ends): scratch_address() looks its device address up once per
// device (the current one) and returns it. moa_step_noalloc puts its
// kernels' partial sums there.
constexpr size_t kScratchBytes = (size_t)64 << 20;
hipError_t scratch_address(void** out);

// Peak microbenchmarks (peaks.hip). read: every byte of [p, p + bytes) once;
// sink needs `grid` words. mfma: grid workgroups of 4 waves, 4 * iters
// 32x32x16 bf16 MFMAs per wave; sink needs grid * 256 floats.
hipError_t launch_peak_read(hipStream_t st, const void* p, size_t bytes, unsigned* sink, int grid);
hipError_t launch_peak_mfma(hipStream_t st, float* sink, int grid, int iters);

}  // namespace moa
