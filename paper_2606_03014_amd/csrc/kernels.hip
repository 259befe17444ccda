// gfx950 (CDNA4) kernels of the ragged MoA generation step.
//
// One engine step runs every co-resident model's rows as one ragged batch:
// rows of the same model are contiguous, and each kernel class is launched
// once per layer for all models (grouped over models), so the weights of each
// active model stream from HBM once per step. The kernels are written for
// 64-wide wavefronts; the dense contractions use the bf16 MFMA
// v_mfma_f32_16x16x32_bf16 with fp32 accumulation.
#include "kernels.h"

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <climits>
#include <cmath>
#include <mutex>

namespace moa {

// Scratch for the kernels of allocation-free calls: partial sums only (every
// byte is written before it is read within a call, so nothing is cleared).
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

hipError_t scratch_address(void** out) {
  static std::mutex mu;
  static void* addr[64] = {};
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess) return err;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}

// Optional event pair attached to the next launch (hipExtLaunchKernel
// timestamps the dispatch itself, so the measured span is the kernel's).
static hipEvent_t g_ev_start = nullptr, g_ev_stop = nullptr;


void set_launch_events(hipEvent_t start, hipEvent_t stop) {
  g_ev_start = start;
  g_ev_stop = stop;
}

template <typename... KArgs, typename... Args>
static void klaunch_shm(void (*kernel)(KArgs...), dim3 grid, dim3 block, unsigned shm, hipStream_t st,
                        Args... args) {
  if (g_ev_start)
    hipExtLaunchKernelGGL(kernel, grid, block, shm, st, g_ev_start, g_ev_stop, 0, args...);
  else
    kernel<<<grid, block, shm, st>>>(args...);
}

template <typename... KArgs, typename... Args>
static void klaunch(void (*kernel)(KArgs...), dim3 grid, dim3 block, hipStream_t st, Args... args) {
  klaunch_shm(kernel, grid, block, 0u, st, args...);
}

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
// (a, b) -> two bf16 in one word (a low), round to nearest even: one
// v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ unsigned pack_bf16(float a, float b) {
  return __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}
// Split-bf16 pair: hi = bf16(a, b); lo = bf16 of the remainders.
__device__ __forceinline__ void split_pair(float a, float b, unsigned& hi, unsigned& lo) {
  hi = pack_bf16(a, b);
  lo = pack_bf16(a - __uint_as_float(hi << 16), b - __uint_as_float(hi & 0xffff0000u));
}

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Split-bf16 store: v ~= hi + lo with hi = bf16(v), lo = bf16(v - hi); the
// pair carries ~16 significant bits, so a GEMM fed hi and lo (two MFMAs per
// weight fragment) sees the fp32 activation almost exactly while the weights
// stay bf16.
__device__ __forceinline__ void store_split(uint16_t* p, size_t lo, size_t i, float v) {
  const uint16_t h = f2bf(v);
  p[i] = h;
  p[i + lo] = f2bf(v - bf2f(h));
}

// Order this wavefront's LDS writes before its later LDS reads (no workgroup barrier).
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

__device__ __forceinline__ const void* pick(const ModelPtrs& mp, int m) {
  const void* r = mp.p[0];
#pragma unroll
  for (int i = 1; i < kMaxModels; ++i)
    if (i == m) r = mp.p[i];
  return r;
}

// Cross-lane moves inside a row of 16 lanes as DPP operand modifiers (plain
// VALU, no LDS crossbar): quad_perm [1,0,3,2] = lane ^ 1, quad_perm [2,3,0,1]
// = lane ^ 2, row_half_mirror = lane 7 - i within each 8 lanes (after the
// two quad steps every lane of a quad holds the quad's value, so the mirror
// brings in the other quad), row_ror:8 = lane ^ 8 within 16 lanes.
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ float sum8(float v) {       // over lanes 8k..8k+7
  v += dpp<0xB1>(v);
  v += dpp<0x4E>(v);
  return v + dpp<0x141>(v);
}
__device__ __forceinline__ float sum16(float v) {      // over lanes 16k..16k+15
  v = sum8(v);
  return v + dpp<0x128>(v);
}
__device__ __forceinline__ float max16(float v) {
  v = fmaxf(v, dpp<0xB1>(v));
  v = fmaxf(v, dpp<0x4E>(v));
  v = fmaxf(v, dpp<0x141>(v));
  return fmaxf(v, dpp<0x128>(v));
}
// lane ^ 16 (within 32 lanes) through ds_swizzle's bit mode
__device__ __forceinline__ float swz_xor16(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x401F));
}

// Sum over the 64 lanes (every lane gets it): DPP within rows of 16, a
// swizzle across the two rows of each half, one exchange across the halves.
__device__ __forceinline__ float wave_sum(float v) {
  v = sum16(v);
  v += swz_xor16(v);
  return v + __shfl_xor(v, 32, 64);
}

// Sum over a 256-thread block; every thread gets the result.
__device__ __forceinline__ float block_sum256(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = red[0] + red[1] + red[2] + red[3];
  __syncthreads();
  return t;
}

// ---------------------------------------------------------------- embedding
// x[t] = E_model[tok] in fp32 (the residual stream is fp32 in every mode).
template <bool BF>
__global__ __launch_bounds__(256) void k_embed(const int* __restrict__ tok_store,
                                               const int* __restrict__ row_tok,
                                               const int* __restrict__ row_model, ModelPtrs embed,
                                               float* __restrict__ x, int d) {
  const int t = blockIdx.x;
  const int tok = tok_store[row_tok[t]];
  const void* E = pick(embed, row_model[t]);
  float* xr = x + (size_t)t * d;
  // 16-byte loads, all of a thread's issued before the first store (d % 256 == 0)
  if (BF) {
    const uint16_t* e = (const uint16_t*)E + (size_t)tok * d;
#pragma unroll 2
    for (int i = threadIdx.x * 8; i < d; i += 256 * 8) {
      const uint4 u = *(const uint4*)(e + i);
      *(float4*)(xr + i) = make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                                       __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
      *(float4*)(xr + i + 4) = make_float4(__uint_as_float(u.z << 16), __uint_as_float(u.z & 0xffff0000u),
                                           __uint_as_float(u.w << 16), __uint_as_float(u.w & 0xffff0000u));
    }
  } else {
    const float* e = (const float*)E + (size_t)tok * d;
#pragma unroll 4
    for (int i = threadIdx.x * 4; i < d; i += 256 * 4) *(float4*)(xr + i) = *(const float4*)(e + i);
  }
}

// ------------------------------------------------- residual add + RMSNorm
// x[r] += sum_s part[s][r] (split-K partial sums of the previous projection),
// out[j] = x[r] * rsqrt(mean(x[r]^2) + eps) * gamma, r = gather ? gather[j] : j.
// One workgroup per row, V4 float4s of the row per thread, thread t owning
// float4s t, t + blockDim, ...: two per thread when d is a multiple of 2048
// (256 threads at d = 2048, 512 at 4096: the smaller workgroup finds room
// beside another stream's kernels sooner, and at 4096 it is as fast alone),
// else one (d / 4 threads, at most 1024).
// The partial-sum loads of a thread are all in flight before they are added.
template <bool BF, int V4>
__global__ __launch_bounds__(1024) void k_add_rmsnorm(float* __restrict__ x, const float* __restrict__ part,
                                                      int nsplit, size_t split_stride,
                                                      const int* __restrict__ gather,
                                                      const int* __restrict__ row_model, ModelPtrs gamma,
                                                      void* __restrict__ out, size_t out_lo, int d, float eps) {
  __shared__ float red[16];
  const int j = blockIdx.x;
  const int r = gather ? gather[j] : j;
  // the row's gain is fetched first, so its dependent loads (model id, gain
  // pointer, gains) overlap the partial-sum loads instead of following the
  // block reduction
  const void* g = pick(gamma, row_model[r]);
  float gv[V4][4];
#pragma unroll
  for (int k = 0; k < V4; ++k) {
    const int i = (threadIdx.x + k * blockDim.x) * 4;
    if (BF) {
      const uint2 gb = *(const uint2*)((const uint16_t*)g + i);
      gv[k][0] = __uint_as_float(gb.x << 16); gv[k][1] = __uint_as_float(gb.x & 0xffff0000u);
      gv[k][2] = __uint_as_float(gb.y << 16); gv[k][3] = __uint_as_float(gb.y & 0xffff0000u);
    } else {
      const float4 gf = *(const float4*)((const float*)g + i);
      gv[k][0] = gf.x; gv[k][1] = gf.y; gv[k][2] = gf.z; gv[k][3] = gf.w;
    }
  }
  float* xrow = x + (size_t)r * d;
  float4 v[V4];
#pragma unroll
  for (int k = 0; k < V4; ++k) v[k] = *(const float4*)(xrow + (threadIdx.x + k * blockDim.x) * 4);
  if (nsplit) {
    const float* prow = part + (size_t)r * d;
#pragma unroll 8
    for (int s = 0; s < nsplit; ++s) {
#pragma unroll
      for (int k = 0; k < V4; ++k) {
        const float4 p = *(const float4*)(prow + (size_t)s * split_stride + (threadIdx.x + k * blockDim.x) * 4);
        v[k].x += p.x; v[k].y += p.y; v[k].z += p.z; v[k].w += p.w;
      }
    }
#pragma unroll
    for (int k = 0; k < V4; ++k) *(float4*)(xrow + (threadIdx.x + k * blockDim.x) * 4) = v[k];
  }
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < V4; ++k) ss += v[k].x * v[k].x + v[k].y * v[k].y + v[k].z * v[k].z + v[k].w * v[k].w;
  ss = wave_sum(ss);
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = ss;
  __syncthreads();
  float tot = 0.f;
  for (int k = 0; k < nw; ++k) tot += red[k];
  const float scale = rsqrtf(tot / (float)d + eps);
#pragma unroll
  for (int k = 0; k < V4; ++k) {
    const int i = (threadIdx.x + k * blockDim.x) * 4;
    const float y[4] = {v[k].x * scale * gv[k][0], v[k].y * scale * gv[k][1], v[k].z * scale * gv[k][2],
                        v[k].w * scale * gv[k][3]};
    if (BF) {
      // split-bf16 pairs packed in hardware, one 8-byte store per plane
      unsigned h01, l01, h23, l23;
      split_pair(y[0], y[1], h01, l01);
      split_pair(y[2], y[3], h23, l23);
      uint16_t* o = (uint16_t*)out + (size_t)j * d + i;
      *(uint2*)o = make_uint2(h01, h23);
      *(uint2*)(o + out_lo) = make_uint2(l01, l23);
    } else {
      *(float4*)((float*)out + (size_t)j * d + i) = make_float4(y[0], y[1], y[2], y[3]);
    }
  }
}

// ------------------------------------------------------------ bf16 GEMMs
// Y = X . W^T for every group (model) of rows, on bf16 MFMA with fp32
// accumulation; X arrives as a split-bf16 pair (hi + lo planes), so each
// weight fragment meets two MFMAs.
//
// Weights are stored tile-shuffled so that one MFMA B-fragment (16 columns x
// 32 k) is 1 KB contiguous, lane-ordered: a wave's weight read is a single
// fully coalesced 1 KB burst per fragment, and a 16-column tile streams
// K*32 bytes contiguously.
//
// 16x16x32 operand layout (lane l of 64): A = rows l%16, k = 8*(l/16)..+8;
// B = column l%16, same k; D = column l%16, rows 4*(l/16)..+4.
//
// --------------------------------------- bf16 GEMM, workgroup-tile variant
// A workgroup (4 wavefronts) owns 16*MT rows x 64*NT columns x one k-split.
// Per stage of 4 MFMA k-steps (128 k) the split-bf16 activation block (both
// planes) is staged in LDS in MFMA A-fragment order (1 KB lane-ordered
// fragments, so every LDS read and write is contiguous) and shared by the four
// wavefronts; each wavefront streams its own NT weight tiles of 16 columns
// from HBM. LDS is double-buffered with one barrier per stage, and the next
// stage's activation and weight loads are issued before the current stage's
// MFMAs, so HBM latency overlaps compute. Workgroup ids are remapped so that
// the row blocks sharing weight tiles run on the same XCD (shared L2).
template <int MT, int NT, int EPI>
__global__ __launch_bounds__(256) void k_gemm_wg(GemmArgs a, int nwg) {
  constexpr int UK = 4;                              // k-steps per stage
  constexpr int UNITS = 2 * MT * UK * 64;            // 16-byte units per stage (both planes)
  constexpr int PER = UNITS / 256;                   // per thread
  __shared__ __align__(16) unsigned char sA[2][UNITS * 16];
  const int per = (nwg + 7) / 8;
  const int blk = (blockIdx.x % 8) * per + blockIdx.x / 8;
  if (blk >= a.total_items) return;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const void* Wg = a.g[0].W;
  int row0 = a.g[0].row0, nrows = a.g[0].nrows, n_mc = a.g[0].n_mc, item0 = a.g[0].item0;
#pragma unroll
  for (int i = 1; i < kMaxGroups; ++i) {
    if (i < a.ngroups && a.g[i].item0 <= blk) {
      Wg = a.g[i].W; row0 = a.g[i].row0; nrows = a.g[i].nrows; n_mc = a.g[i].n_mc; item0 = a.g[i].item0;
    }
  }
  const int idx = blk - item0;
  const int mc = idx % n_mc;
  const int rest = idx / n_mc;
  const int s = rest % a.S;
  const int nb = rest / a.S;
  const int ks0 = s * a.ksteps;
  const int nt0 = (nb * 4 + w) * NT;                 // this wavefront's first 16-column tile
  const int KS = a.K >> 5;
  const u32x4* wp = (const u32x4*)Wg + ((size_t)nt0 * KS + ks0) * 64 + lane;
  const size_t wt = (size_t)KS * 64;                 // u32x4 distance between tiles
  const int rbase = row0 + mc * MT * 16;
  const int rend = row0 + nrows;

  // Staging: unit u = t + 256*i is lane ln = u % 64 of fragment (plane p,
  // m-tile mt, k-step ku) = (u / (MT*UK*64), (u / (UK*64)) % MT, (u / 64) % UK):
  // row 16*mt + ln % 16, k = 32*ku + 8*(ln / 16) .. +8 of that plane.
  const uint16_t* X = (const uint16_t*)a.X;
  size_t xoff[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int u = threadIdx.x + 256 * i;
    const int ln = u & 63, ku = (u >> 6) % UK, mt = (u / (UK * 64)) % MT, p = u / (MT * UK * 64);
    const int r = min(rbase + mt * 16 + (ln & 15), rend - 1);
    xoff[i] = (size_t)p * a.x_lo + (size_t)r * a.K + (size_t)ks0 * 32 + ku * 32 + (ln >> 4) * 8;
  }

  f32x4_t acc[MT][NT];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[m][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  u32x4 stg[PER], b[UK][NT];
#pragma unroll
  for (int i = 0; i < PER; ++i) stg[i] = *(const u32x4*)(X + xoff[i]);
#pragma unroll
  for (int u = 0; u < UK; ++u)
#pragma unroll
    for (int j = 0; j < NT; ++j) b[u][j] = wp[j * wt + u * 64];
#pragma unroll
  for (int i = 0; i < PER; ++i) *(u32x4*)(sA[0] + (threadIdx.x + 256 * i) * 16) = stg[i];
  __syncthreads();

  const int nstage = a.ksteps / UK;
  for (int st = 0; st < nstage; ++st) {
    const int cur = st & 1;
    const bool more = st + 1 < nstage;
    u32x4 bn[UK][NT];
    if (more) {                                       // next stage: activations and weights
      const size_t ko = (size_t)(st + 1) * UK * 32;
#pragma unroll
      for (int i = 0; i < PER; ++i) stg[i] = *(const u32x4*)(X + xoff[i] + ko);
#pragma unroll
      for (int u = 0; u < UK; ++u)
#pragma unroll
        for (int j = 0; j < NT; ++j) bn[u][j] = wp[j * wt + ((st + 1) * UK + u) * 64];
    }
    const unsigned char* A = sA[cur];
#pragma unroll
    for (int u = 0; u < UK; ++u) {
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const u32x4 ah = *(const u32x4*)(A + ((0 * MT + m) * UK + u) * 1024 + lane * 16);
#pragma unroll
        for (int j = 0; j < NT; ++j)
          acc[m][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, ah),
                                                              __builtin_bit_cast(bf16x8_t, b[u][j]), acc[m][j], 0, 0, 0);
      }
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const u32x4 al = *(const u32x4*)(A + ((1 * MT + m) * UK + u) * 1024 + lane * 16);
#pragma unroll
        for (int j = 0; j < NT; ++j)
          acc[m][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, al),
                                                              __builtin_bit_cast(bf16x8_t, b[u][j]), acc[m][j], 0, 0, 0);
      }
    }
    if (more) {
#pragma unroll
      for (int i = 0; i < PER; ++i) *(u32x4*)(sA[cur ^ 1] + (threadIdx.x + 256 * i) * 16) = stg[i];
#pragma unroll
      for (int u = 0; u < UK; ++u)
#pragma unroll
        for (int j = 0; j < NT; ++j) b[u][j] = bn[u][j];
    }
    __syncthreads();
  }

  const int col = lane & 15;
  const int rq = (lane >> 4) * 4;
  if (EPI == EPI_F32) {
    float* out = a.out + (size_t)s * a.out_split;
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = rbase + m * 16 + rq + i;
          if (r < rend) out[(size_t)r * a.N + (nt0 + j) * 16 + col] = acc[m][j][i];
        }
  } else {
    const int half = a.N >> 1;
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int p = 0; p < NT / 2; ++p)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = rbase + m * 16 + rq + i;
          if (r < rend) {
            const float g = acc[m][2 * p][i], u = acc[m][2 * p + 1][i];
            store_split(a.hout, a.h_lo, (size_t)r * half + ((nt0 >> 1) + p) * 16 + col, g / (1.f + __expf(-g)) * u);
          }
        }
  }
}

// ---------------------------------------- wait, LDS and direct-load helpers
// Explicit waits, LDS addressing and untracked LDS reads shared by the GEMM
// and attention kernels below. Direct global->LDS loads
// (global_load_lds_dwordx4) move one 1 KB MFMA fragment per instruction.
template <int N> __device__ __forceinline__ void wait_vmcnt() {
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }
#define MOA_LDS(p) ((__attribute__((address_space(3))) void*)(p))
// 32-bit LDS address of a pointer into shared memory
__device__ __forceinline__ unsigned lds_addr(const void* p) {
  return (unsigned)(size_t)(const __attribute__((address_space(3))) void*)p;
}
// Two 8-byte LDS reads at addr + 8*O0 and addr + 8*O1 into one register
// quad. The compiler does not track it: pair it with lgkm_wait_for().
template <int O0, int O1>
__device__ __forceinline__ u32x4 ds_read2_b64(unsigned addr) {
  u32x4 v;
  asm volatile("ds_read2_b64 %0, %1 offset0:%2 offset1:%3" : "=v"(v) : "v"(addr), "i"(O0), "i"(O1));
  return v;
}
// Two transposed 8-byte LDS reads (ds_read_b64_tr_b16) at addr + O0 and
// addr + O1 into one register quad; untracked like ds_read2_b64 above.
template <int O0, int O1>
__device__ __forceinline__ u32x4 ds_read_tr16_pair(unsigned addr) {
  u32x2_t a, b;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(a) : "v"(addr), "i"(O0));
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(b) : "v"(addr), "i"(O1));
  return u32x4{a.x, a.y, b.x, b.y};
}
// One 4-byte LDS store the compiler does not track (ordered by "memory" and by
// the explicit LDS waits before each barrier).
__device__ __forceinline__ void ds_write_b32(unsigned addr, unsigned v) {
  asm volatile("ds_write_b32 %0, %1" : : "v"(addr), "v"(v) : "memory");
}
// Wait for every outstanding LDS access; tying v makes its later uses follow.
__device__ __forceinline__ void lgkm_wait_for(u32x4& v) { asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(v)); }

// ----------------------------- medium- and large-M GEMM (16x16x32 MFMA)
// From a few dozen rows per model up to prefill chunks of many thousands.
// At decode sizes every weight byte feeds only that many rows of MFMA work,
// so the GEMM must stream the weights at HBM speed; at prefill sizes it is
// bound by the matrix cores, and keeping the weights out of LDS leaves the
// LDS to the activations. A workgroup of NW waves owns one row chunk of a
// group (mrows rows, at most 16*RT: a group of up to that many rows is one
// chunk, so each weight tile leaves HBM once per step; a larger group is cut
// into chunks whose items for one column block run side by side on one XCD)
// x NW * CT * 16 columns x one k-split.
//  * The split-bf16 activation block of a 32-k stage (2*RT fragments of 1 KB,
//    both planes) is shared by the waves: it goes HBM/L2 -> LDS by direct
//    loads into a ring of D + 1 slots.
//  * Each wave streams its own CT weight tiles (1 KB fragments) straight into
//    a register ring D stages deep (a stage's loads are issued once its
//    registers have fed the MFMAs: issuing them before, from a ring one
//    stage deeper, measured ~10% slower at 100+ rows), so the LDS holds only
//    activations: the planner sizes the grid to the resident slots
//    (a grid of more items than slots ran at half the streaming rate in its
//    last, partly empty round).
//  * Per stage a wave reads its hi-plane fragments, multiplies them, then the
//    lo plane (other waves on the SIMD fill the read latency); the RT x CT
//    accumulators form that many independent MFMA chains (16x16x32 needs
//    about 16 to reach its rate).
//  * Loads complete in issue order: stage s's activation loads, then its
//    weight loads, so waiting until D - 1 stages' worth of loads are
//    outstanding makes stage s resident.
//  * k-splits take KS / S k-steps each, rounded (any S).
// N 16-byte LDS reads at addr + OFF + 1024 * i and the wait for them, in
// one asm statement: the compiler sees the registers only once they hold
// the data (an asm read whose wait came later let it copy a register that
// was still in flight when registers were scarce).
template <int N, int OFF>
__device__ __forceinline__ void lds_frags(u32x4 (&v)[N], unsigned addr) {
  static_assert(N == 2 || N == 4 || N == 8, "fragment count");
  if constexpr (N == 2) {
    asm volatile("ds_read_b128 %0, %2 offset:%3\n\tds_read_b128 %1, %2 offset:%4\n\ts_waitcnt lgkmcnt(0)"
                 : "=&v"(v[0]), "=&v"(v[1]) : "v"(addr), "i"(OFF), "i"(OFF + 1024));
  } else if constexpr (N == 4) {
    asm volatile("ds_read_b128 %0, %4 offset:%5\n\tds_read_b128 %1, %4 offset:%6\n\t"
                 "ds_read_b128 %2, %4 offset:%7\n\tds_read_b128 %3, %4 offset:%8\n\ts_waitcnt lgkmcnt(0)"
                 : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3])
                 : "v"(addr), "i"(OFF), "i"(OFF + 1024), "i"(OFF + 2048), "i"(OFF + 3072));
  } else {
    asm volatile("ds_read_b128 %0, %8 offset:%9\n\tds_read_b128 %1, %8 offset:%10\n\t"
                 "ds_read_b128 %2, %8 offset:%11\n\tds_read_b128 %3, %8 offset:%12\n\t"
                 "ds_read_b128 %4, %8 offset:%13\n\tds_read_b128 %5, %8 offset:%14\n\t"
                 "ds_read_b128 %6, %8 offset:%15\n\tds_read_b128 %7, %8 offset:%16\n\ts_waitcnt lgkmcnt(0)"
                 : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5]), "=&v"(v[6]),
                   "=&v"(v[7])
                 : "v"(addr), "i"(OFF), "i"(OFF + 1024), "i"(OFF + 2048), "i"(OFF + 3072), "i"(OFF + 4096),
                   "i"(OFF + 5120), "i"(OFF + 6144), "i"(OFF + 7168));
  }
}

template <int RT, int CT, int NW, int D, int EPI>
__global__ __launch_bounds__(64 * NW) void k_gemm_mm(GemmArgs a, int nwg) {
  constexpr int P = D + 1;
  constexpr int FA = 2 * RT;                         // activation fragments per stage (plane, row tile)
  constexpr int DPW = FA / NW;                       // activation loads per wave per stage
  static_assert(FA % NW == 0, "activation fragments per wave");
  constexpr int PER = DPW + CT;                      // loads per wave per stage
  constexpr unsigned SLOT = FA * 1024;
  extern __shared__ __align__(1024) unsigned char smem[];
  const int per = (nwg + 7) / 8;
  const int blk = (blockIdx.x % 8) * per + blockIdx.x / 8;
  if (blk >= a.total_items) return;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const void* Wg = a.g[0].W;
  int row0 = a.g[0].row0, nrows = a.g[0].nrows, n_mc = a.g[0].n_mc, item0 = a.g[0].item0, mrows = a.g[0].mrows;
#pragma unroll
  for (int i = 1; i < kMaxGroups; ++i) {
    if (i < a.ngroups && a.g[i].item0 <= blk) {
      Wg = a.g[i].W; row0 = a.g[i].row0; nrows = a.g[i].nrows; n_mc = a.g[i].n_mc; item0 = a.g[i].item0;
      mrows = a.g[i].mrows;
    }
  }
  // items of a group: ((split, column block), row chunk), row chunks
  // fastest: the chunks of one weight column block are neighbours, so they
  // run together on one XCD and its L2 serves the block to all of them
  const int ncol = a.N / (NW * CT * 16);
  const int idx = blk - item0;
  const int mc = idx % n_mc;
  const int nb = (idx / n_mc) % ncol;
  const int s = idx / (n_mc * ncol);
  const int KS = a.K >> 5;
  const int ks0 = (s * KS) / a.S, nk = ((s + 1) * KS) / a.S - ks0;
  const int crows = mrows > 0 ? mrows : RT * 16;
  const int rbase = row0 + mc * crows;
  const int rend = min(row0 + nrows, rbase + crows);  // this chunk's rows end
  const int nrt = min(RT, (rend - rbase + 15) >> 4); // row tiles holding rows (the rest are padding:
                                                     // still loaded, so every wave's load count per
                                                     // stage stays PER, but neither read nor multiplied)
  const int nt0 = (nb * NW + w) * CT;                // this wave's first 16-column weight tile

  const unsigned char* asrc[DPW];
#pragma unroll
  for (int i = 0; i < DPW; ++i) {
    const int f = w * DPW + i;
    const int p = f / RT, r = f % RT;
    const int row = min(rbase + 16 * r + (lane & 15), rend - 1);
    asrc[i] = (const unsigned char*)((const uint16_t*)a.X + (size_t)p * a.x_lo + (size_t)row * a.K +
                                     (size_t)ks0 * 32 + 8 * (lane >> 4));
  }
  const u32x4* bsrc = (const u32x4*)Wg + ((size_t)nt0 * KS + ks0) * 64 + lane;
  const size_t btile = (size_t)KS * 64;              // u32x4 between weight tiles
  // Every stage issues the same loads, past the last stage too (clamped to
  // it; those activation copies land in ring slots nobody reads again and
  // the weight copies are dropped), so the number of loads in flight is the
  // same at every wait and the compiler never has to drain the whole queue
  // to make a register of the ring safe to read.
  auto issueA = [&](int st) {
    const int sk = min(st, nk - 1);
    unsigned char* sl = smem + (st % P) * SLOT;
#pragma unroll
    for (int i = 0; i < DPW; ++i)
      __builtin_amdgcn_global_load_lds((const void*)(asrc[i] + (size_t)sk * 64), MOA_LDS(sl + (w * DPW + i) * 1024),
                                       16, 0, 0);
  };
  auto loadB = [&](int st, u32x4* dst) {
    const size_t sk = (size_t)min(st, nk - 1) * 64;
#pragma unroll
    for (int c = 0; c < CT; ++c) dst[c] = bsrc[c * btile + sk];
  };

  f32x4_t acc[RT][CT];
#pragma unroll
  for (int r = 0; r < RT; ++r)
#pragma unroll
    for (int c = 0; c < CT; ++c) acc[r][c] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  u32x4 breg[D][CT];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    issueA(d);
    loadB(d, breg[d]);
  }
  const unsigned lbase = lds_addr(smem) + lane * 16;
  for (int st0 = 0; st0 < nk; st0 += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int st = st0 + d;
      // stage st resident (D - 1 newer stages in flight); every wave done
      // with stage st - 1, whose slot is refilled next
      wait_vmcnt<(D - 1) * PER>();
      wait_lgkm0();
      asm volatile("s_barrier" ::: "memory");
      issueA(st + D);
      if (st < nk) {
        const unsigned sb = lbase + (unsigned)(st % P) * SLOT;
        u32x4 ah[RT], al[RT];
        lds_frags<RT, 0>(ah, sb);
#pragma unroll
        for (int r = 0; r < RT; ++r)
          if (r < nrt) {
#pragma unroll
            for (int c = 0; c < CT; ++c)
              acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, ah[r]),
                                                                  __builtin_bit_cast(bf16x8_t, breg[d][c]), acc[r][c], 0, 0, 0);
          }
        lds_frags<RT, RT * 1024>(al, sb);
#pragma unroll
        for (int r = 0; r < RT; ++r)
          if (r < nrt) {
#pragma unroll
            for (int c = 0; c < CT; ++c)
              acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, al[r]),
                                                                  __builtin_bit_cast(bf16x8_t, breg[d][c]), acc[r][c], 0, 0, 0);
          }
      }
      loadB(st + D, breg[d]);
    }
  }
  wait_vmcnt<0>();                                   // no load may land in LDS after the workgroup ends

  const int col = lane & 15;
  const int rq = (lane >> 4) * 4;
  if (EPI == EPI_F32) {
    float* out = a.out + (size_t)s * a.out_split;
#pragma unroll
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int c = 0; c < CT; ++c)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = rbase + r * 16 + rq + i;
          if (row < rend) out[(size_t)row * a.N + (nt0 + c) * 16 + col] = acc[r][c][i];
        }
  } else {
    // tiles (2p, 2p+1) are (gate, up) of the same 16 hidden units
    const int half = a.N >> 1;
#pragma unroll
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int q = 0; q < CT / 2; ++q)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = rbase + r * 16 + rq + i;
          if (row < rend) {
            const float g = acc[r][2 * q][i], u = acc[r][2 * q + 1][i];
            store_split(a.hout, a.h_lo, (size_t)row * half + ((nt0 >> 1) + q) * 16 + col, g / (1.f + __expf(-g)) * u);
          }
        }
  }
}

// ------------------------------------------------------------ fp32 GEMM
// Plain fp32 FMA GEMM for the fp32 engine mode: a workgroup computes 16 rows
// x 64 columns; W is row-major [N][K].
__global__ __launch_bounds__(256) void k_gemm_f32(GemmArgs a) {
  const int item = blockIdx.x;
  const void* Wg = a.g[0].W;
  int row0 = a.g[0].row0, nrows = a.g[0].nrows, n_mc = a.g[0].n_mc, item0 = a.g[0].item0;
#pragma unroll
  for (int i = 1; i < kMaxGroups; ++i) {
    if (i < a.ngroups && a.g[i].item0 <= item) {
      Wg = a.g[i].W; row0 = a.g[i].row0; nrows = a.g[i].nrows; n_mc = a.g[i].n_mc; item0 = a.g[i].item0;
    }
  }
  const int idx = item - item0;
  const int mc = idx % n_mc, nb = idx / n_mc;
  const int colw = nb * 64 + (threadIdx.x & 63);
  const int rb = row0 + mc * 16 + (threadIdx.x >> 6) * 4;
  const int rend = row0 + nrows;
  const float* W = (const float*)Wg + (size_t)colw * a.K;
  const float* X = (const float*)a.X;
  const float* xr[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) xr[i] = X + (size_t)min(rb + i, rend - 1) * a.K;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < a.K; ++k) {
    const float w = W[k];
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = fmaf(xr[i][k], w, acc[i]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (rb + i < rend) a.out[(size_t)(rb + i) * a.N + colw] = acc[i];
}

// h = silu(gate) * up for the fp32 mode; gu rows are [gate(ffn) | up(ffn)].
__global__ __launch_bounds__(256) void k_swiglu_f32(const float* __restrict__ gu, float* __restrict__ h,
                                                    int ffn) {
  const int t = blockIdx.x;
  const float* r = gu + (size_t)t * 2 * ffn;
  for (int i = threadIdx.x; i < ffn; i += 256) {
    const float g = r[i];
    h[(size_t)t * ffn + i] = g / (1.f + expf(-g)) * r[ffn + i];
  }
}

// ------------------------------------------------------ RoPE + KV append
// Reduces the QKV partial sums, rotates q and k (pairs (i, i + hd/2) turned by
// pos * theta^(-2i/hd), table precomputed in fp64 and rounded to fp32), stores
// q (fp32), and writes k, v (rounded to the cache type) into the row's paged-KV slot: block bt[pos / 16], slot
// pos % 16. Pool layout: [layer][block][kv_head][K|V][16][hd].
template <bool BF>
__global__ __launch_bounds__(256) void k_rope_kv(const float* __restrict__ part, int nsplit, size_t split_stride,
                                                 const int* __restrict__ row_pos, const int* __restrict__ row_bt,
                                                 const int* __restrict__ bt_store, const float2* __restrict__ tab,
                                                 float* __restrict__ qv, void* __restrict__ kvv, int layer, int NB,
                                                 int n_h, int n_kv, int hd) {
  // work items of a row: (n_h + n_kv) * hd/2 rotation pairs, then n_kv * hd v elements
  const int t = blockIdx.x;
  const int item = blockIdx.y * 256 + threadIdx.x;
  const int half = hd >> 1;
  const int npairs = (n_h + n_kv) * half;
  if (item >= npairs + n_kv * hd) return;
  const int pos = row_pos[t];
  const int qkv = (n_h + 2 * n_kv) * hd;
  const float* pr = part + (size_t)t * qkv;
  const int blk = bt_store[row_bt[t] + (pos >> 4)];
  const int off = pos & 15;
  const size_t hs = (size_t)2 * kBlock * hd;
  const size_t lbase = ((size_t)layer * NB + blk) * n_kv * hs;
  if (item < npairs) {
    const int head = item / half, jj = item - head * half;
    const int c = head * hd + jj;
    const float2 cs = tab[(size_t)pos * half + jj];   // in flight with the partial sums
    float x1 = 0.f, x2 = 0.f;
#pragma unroll 16
    for (int s = 0; s < nsplit; ++s) {
      x1 += pr[(size_t)s * split_stride + c];
      x2 += pr[(size_t)s * split_stride + c + half];
    }
    const float y1 = x1 * cs.x - x2 * cs.y;
    const float y2 = x2 * cs.x + x1 * cs.y;
    if (head < n_h) {
      const size_t o = ((size_t)t * n_h + head) * hd + jj;
      qv[o] = y1;
      qv[o + half] = y2;
    } else {
      const size_t o = lbase + (size_t)(head - n_h) * hs + off * hd + jj;
      if (BF) { ((uint16_t*)kvv)[o] = f2bf(y1); ((uint16_t*)kvv)[o + half] = f2bf(y2); }
      else { ((float*)kvv)[o] = y1; ((float*)kvv)[o + half] = y2; }
    }
  } else {
    const int i = item - npairs;
    const int kh = i / hd, dd = i - kh * hd;
    const int c = (n_h + n_kv) * hd + i;
    float v = 0.f;
#pragma unroll 16
    for (int s = 0; s < nsplit; ++s) v += pr[(size_t)s * split_stride + c];
    const size_t o = lbase + (size_t)kh * hs + kBlock * hd + off * hd + dd;
    if (BF) ((uint16_t*)kvv)[o] = f2bf(v);
    else ((float*)kvv)[o] = v;
  }
}

// ------------------------------------------------ paged attention (split-KV)
// One workgroup = one query row x one KV head x one key range [k0, k1); its
// GQ wavefronts are the GQ query heads that share the KV head, so each K/V
// tile is read from HBM once for the whole group. The range's block ids are
// first copied to LDS (dynamic shared memory sized by the host), then tiles
// of 64 keys are staged in LDS with 16-byte coalesced loads (a 16-slot block
// of one KV head is contiguous); the next tile's loads are issued into
// registers before the current tile is computed. In a tile, lane l owns key
// 8*p + l/8 (p = 0..7) and head-dim chunk l%8: q.k partial dots are combined
// across the 8 lanes of a key with xor-shuffles, the tile max across the
// wavefront with shuffles, and P.V accumulates per lane on its own keys and
// dims (combined once at the end). Softmax runs in base 2 on scores
// pre-scaled by log2(e)/sqrt(hd).
#ifndef ATTN_WPE
#define ATTN_WPE 1
#endif
template <int HD, int GQ, bool BF, int TK>
__global__ __launch_bounds__(GQ * 64, ATTN_WPE) void k_attn(const AttnItem* __restrict__ items, const float* __restrict__ qv,
                                                  const void* __restrict__ kvv, const int* __restrict__ bt_store,
                                                  const int* __restrict__ row_bt, int layer, int NB, int n_h,
                                                  int n_kv, float scale_log2, void* __restrict__ outv,
                                                  size_t out_lo, float* __restrict__ pacc, float* __restrict__ pml) {
  constexpr int CH = HD / 8;
  constexpr int ESZ = BF ? 2 : 4;
  constexpr int ROWB = HD * ESZ;
  constexpr int CPR = ROWB / 16;                 // 16-byte chunks per key row
  constexpr int NCH = 2 * TK * CPR;              // chunks per tile (K and V)
  constexpr int NT = GQ * 64;
  constexpr int PER = (NCH + NT - 1) / NT;       // chunks per thread
  __shared__ __align__(16) unsigned char sK[TK * ROWB];
  __shared__ __align__(16) unsigned char sV[TK * ROWB];
  extern __shared__ unsigned long long sbo[];    // byte offsets of the key range's blocks in the layer's pool

  const AttnItem it = items[blockIdx.x];
  const int kvh = blockIdx.y;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g8 = lane >> 3, c8 = lane & 7;
  const int h = kvh * GQ + w;

  const size_t hs = (size_t)2 * kBlock * HD;     // elements per (block, kv head)
  const unsigned char* pool = (const unsigned char*)kvv + ((size_t)layer * NB * n_kv + kvh) * hs * ESZ;
  const unsigned long long blk_stride = (unsigned long long)n_kv * hs * ESZ;
  const int b0 = it.k0 >> 4, nb = ((it.k1 - 1) >> 4) - b0 + 1;
  {
    const int* bt = bt_store + it.bt_off;
    for (int i = threadIdx.x; i < nb; i += NT) sbo[i] = (unsigned long long)bt[i] * blk_stride;
  }
  // bf16 cache: q enters the dot products as a split-bf16 pair (hi + lo,
  // pre-scaled by log2(e)/sqrt(hd)) through v_dot2_f32_bf16, which multiplies
  // bf16 pairs exactly and accumulates in fp32; fp32 cache: plain fp32 q.
  float q[BF ? 1 : CH];
  unsigned qh[BF ? CH / 2 : 1], ql[BF ? CH / 2 : 1];
  {
    const size_t qo = ((size_t)it.row * n_h + h) * HD + c8 * CH;
    if (BF) {
#pragma unroll
      for (int i = 0; i < CH / 2; ++i)
        split_pair(qv[qo + 2 * i] * scale_log2, qv[qo + 2 * i + 1] * scale_log2, qh[i], ql[i]);
    } else {
#pragma unroll
      for (int i = 0; i < CH; ++i) q[i] = qv[qo + i];
    }
  }
  float m = -INFINITY, l = 0.f, acc[CH];
#pragma unroll
  for (int i = 0; i < CH; ++i) acc[i] = 0.f;

  // loop-invariant part of every chunk this thread moves: key in the tile,
  // byte offset inside its 16-slot block, LDS destination
  int ckey[PER];
  unsigned coff[PER];
  unsigned char* cdst[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int c = min((int)threadIdx.x + j * NT, NCH - 1);
    const int isV = c / (TK * CPR);
    const int rem = c - isV * (TK * CPR);
    const int key = rem / CPR, cc = rem - key * CPR;
    ckey[j] = (threadIdx.x + j * NT < NCH) ? key : (1 << 29);     // out-of-tile chunks never load
    coff[j] = (unsigned)((isV * kBlock * HD + (key & 15) * HD) * ESZ + cc * 16);
    cdst[j] = (isV ? sV : sK) + rem * 16;
  }
  __syncthreads();

  uint4 pre[PER];
  auto fetch = [&](int t0) {
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int p = t0 + ckey[j];
      uint4 val = make_uint4(0u, 0u, 0u, 0u);
      if (p < it.k1) val = *(const uint4*)(pool + sbo[(p >> 4) - b0] + coff[j]);
      pre[j] = val;
    }
  };
  fetch(it.k0);
  for (int t0 = it.k0; t0 < it.k1; t0 += TK) {
#pragma unroll
    for (int j = 0; j < PER; ++j)
      if (threadIdx.x + j * NT < NCH) *(uint4*)cdst[j] = pre[j];
    __syncthreads();
    if (t0 + TK < it.k1) fetch(t0 + TK);

    constexpr int NP = TK / 8;                   // keys per lane group
    float s[NP];
#pragma unroll
    for (int p8 = 0; p8 < NP; ++p8) {
      const int key = p8 * 8 + g8;
      float dot = 0.f;
      if (BF) {
        const unsigned* kr = (const unsigned*)(sK + key * ROWB + c8 * CH * 2);
#pragma unroll
        for (int i = 0; i < CH / 2; ++i) {
          const bf16x2_t kp = __builtin_bit_cast(bf16x2_t, kr[i]);
          dot = __builtin_amdgcn_fdot2_f32_bf16(kp, __builtin_bit_cast(bf16x2_t, qh[i]), dot, false);
          dot = __builtin_amdgcn_fdot2_f32_bf16(kp, __builtin_bit_cast(bf16x2_t, ql[i]), dot, false);
        }
        dot = sum8(dot);
      } else {
        const float* kr = (const float*)(sK + key * ROWB) + c8 * CH;
#pragma unroll
        for (int i = 0; i < CH; ++i) dot = fmaf(q[i], kr[i], dot);
        dot = sum8(dot) * scale_log2;
      }
      s[p8] = (t0 + key < it.k1) ? dot : -INFINITY;
    }
    float mx = s[0];
#pragma unroll
    for (int p8 = 1; p8 < NP; ++p8) mx = fmaxf(mx, s[p8]);
    mx = fmaxf(mx, dpp<0x128>(mx));
    mx = fmaxf(mx, swz_xor16(mx));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float mnew = fmaxf(m, mx);
    const float alpha = __builtin_amdgcn_exp2f(m - mnew);
    l *= alpha;
#pragma unroll
    for (int i = 0; i < CH; ++i) acc[i] *= alpha;
#pragma unroll
    for (int p8 = 0; p8 < NP; ++p8) {
      const float pj = __builtin_amdgcn_exp2f(s[p8] - mnew);
      l += pj;
      const int key = p8 * 8 + g8;
      if (BF) {
        const uint16_t* vr = (const uint16_t*)(sV + key * ROWB) + c8 * CH;
#pragma unroll
        for (int i = 0; i < CH; ++i) acc[i] = fmaf(pj, bf2f(vr[i]), acc[i]);
      } else {
        const float* vr = (const float*)(sV + key * ROWB) + c8 * CH;
#pragma unroll
        for (int i = 0; i < CH; ++i) acc[i] = fmaf(pj, vr[i], acc[i]);
      }
    }
    m = mnew;
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    acc[i] += __shfl_xor(acc[i], 8, 64);
    acc[i] += __shfl_xor(acc[i], 16, 64);
    acc[i] += __shfl_xor(acc[i], 32, 64);
  }
  l += __shfl_xor(l, 8, 64);
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  if (g8 == 0) {
    if (it.slot < 0) {
      const float inv = 1.f / l;
      const size_t o = ((size_t)it.row * n_h + h) * HD + c8 * CH;
#pragma unroll
      for (int i = 0; i < CH; ++i) {
        if (BF) store_split((uint16_t*)outv, out_lo, o + i, acc[i] * inv);
        else ((float*)outv)[o + i] = acc[i] * inv;
      }
    } else {
      const size_t o = ((size_t)it.slot * n_h + h) * HD + c8 * CH;
#pragma unroll
      for (int i = 0; i < CH; ++i) pacc[o + i] = acc[i];
      if (c8 == 0) {
        pml[((size_t)it.slot * n_h + h) * 2] = m;
        pml[((size_t)it.slot * n_h + h) * 2 + 1] = l;
      }
    }
  }
}

// ------------------------------------------ causal prefill attention (MFMA)
// Causal prefill attention on the 32x32x16 MFMA. A workgroup is one query
// head and up to kPrefillRows consecutive positions of one request, four
// wavefronts of 32 query rows each; key tiles of 32 keys cover [0, pos0 + nq).
// Scores are formed transposed, S^T = K Q^T (A = K tile, B = the wave's q
// rows), so lane l of a wave holds the 16 scores of query row l%32 for keys
// 8(e/4) + 4(l/32) + e%4 of the tile: the online softmax is per lane (plus
// one exchange with lane l^32), and those 16 probabilities are directly the
// B operand of O^T = V^T P^T, with the key order inside each 16-key step
// permuted identically in A (V^T, read from LDS) and B (P^T, in registers).
// q and P enter the MFMAs as split bf16 (hi + lo, two MFMAs each). K tiles
// reach LDS by direct global->LDS loads into a three-stage ring, in MFMA
// fragment order; V tiles go through registers and are stored transposed.
#ifndef PREFILL_WPE
#define PREFILL_WPE 2
#endif
template <int HD>
__global__ __launch_bounds__(256, PREFILL_WPE) void k_prefill_attn(const PrefillItem* __restrict__ items,
                                                      const float* __restrict__ qv, const uint16_t* __restrict__ kv,
                                                      const int* __restrict__ bt_store, int layer, int NB, int n_h,
                                                      int n_kv, float scale_log2, uint16_t* __restrict__ out,
                                                      size_t out_lo) {
  constexpr int TK = 32;                    // keys per tile
  constexpr int DS = HD / 16;               // 16-wide dim steps of S^T = K Q^T
  constexpr int DT = HD / 32;               // 32-dim tiles of O^T
  constexpr int KFR = DS;                   // K fragments (1 KB) per tile
  constexpr int KPW = KFR / 4;              // K fragments loaded per wave
  constexpr int ROWB = HD * 2;              // bytes per V row
  constexpr int CPR = ROWB / 16;            // 16-byte chunks per V row
  constexpr int KPF = 1024 / ROWB;          // V rows per 1 KB fragment
  constexpr int VFR = TK * ROWB / 1024;     // V fragments per tile
  constexpr int VPW = VFR / 4;              // V fragments loaded per wave
  constexpr int NKS = 3;                    // ring stages (K and V)
  static_assert(KPW >= 1 && KPW * 4 == KFR && VPW >= 1 && VPW * 4 == VFR, "tile shape");
  // One dynamic LDS block (sized by the launcher): the K ring (NKS x KFR KB),
  // the V ring (NKS x VFR KB), then the block ids of keys [0, kmax).
  extern __shared__ __align__(1024) unsigned char sKd[];
  unsigned char* sV = sKd + NKS * KFR * 1024;
  int* sbt = (int*)(sV + NKS * VFR * 1024);

  const PrefillItem it = items[blockIdx.x];
  const int h = blockIdx.y;
  const int kvh = h / (n_h / n_kv);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c32 = lane & 31, hf = lane >> 5;
  const int kmax = it.pos0 + it.nq;          // keys [0, kmax)
  const int ntile = (kmax + TK - 1) / TK;
  const size_t hs = (size_t)2 * kBlock * HD;
  const uint16_t* pool = kv + ((size_t)layer * NB * n_kv + kvh) * hs;
  const size_t bstride = (size_t)n_kv * hs;
  // The block ids live in LDS for the whole item: a K/V address then never
  // waits on a global load, which (vector loads complete in order) would also
  // wait for every tile already in flight.
  {
    const int* bt = bt_store + it.bt_off;
    const int nblk = (kmax + kBlock - 1) / kBlock;
    for (int i = threadIdx.x; i < nblk; i += 256) sbt[i] = bt[i];
    __syncthreads();
  }

  // B operand of S^T: query row 32w + l%32 (rows past nq read row nq-1 and
  // are never stored), dims 16s + 8(l/32) .. +8, scaled to log2 units, split
  u32x4 qh[DS], ql[DS];
  {
    const int r = min(32 * w + c32, it.nq - 1);
    const float* qrow = qv + ((size_t)(it.row0 + r) * n_h + h) * HD + 8 * hf;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      unsigned hv[4], lv[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        split_pair(qrow[16 * s + 2 * j] * scale_log2, qrow[16 * s + 2 * j + 1] * scale_log2, hv[j], lv[j]);
      qh[s] = u32x4{hv[0], hv[1], hv[2], hv[3]};
      ql[s] = u32x4{lv[0], lv[1], lv[2], lv[3]};
    }
  }
  const int qpos = it.pos0 + 32 * w + c32;   // this lane's query position

  // Tile t of K and V, both by direct loads into their rings (slot t % NKS).
  // K fragment s holds key t*32 + l%32, dims 16s + 8(l/32) .. +8 in lane l.
  // V keeps its natural [key][dim] rows; the 16-byte chunk c of row r sits at
  // chunk position c ^ 2(r % 4), so the four rows a transposed read touches
  // fall on different LDS banks.
  const int vrow_in = lane / CPR, vcp = lane % CPR;
  auto issue_kv = [&](int t) {
    {
      const int key = min(t * TK + c32, kmax - 1);
      const uint16_t* base = pool + (size_t)sbt[key >> 4] * bstride + (key & 15) * HD + 8 * hf;
      unsigned char* sl = sKd + (t % NKS) * KFR * 1024;
#pragma unroll
      for (int i = 0; i < KPW; ++i) {
        const int s = w * KPW + i;
        __builtin_amdgcn_global_load_lds((const void*)(base + 16 * s), MOA_LDS(sl + s * 1024), 16, 0, 0);
      }
    }
    unsigned char* vs = sV + (t % NKS) * VFR * 1024;
#pragma unroll
    for (int i = 0; i < VPW; ++i) {
      const int f = w * VPW + i;
      const int r = f * KPF + vrow_in;                    // row of the tile this lane fills
      const int key = min(t * TK + r, kmax - 1);
      const int gc = vcp ^ ((r & 3) << 1);                // chunk of the key's row it brings
      const uint16_t* src = pool + (size_t)sbt[key >> 4] * bstride + kBlock * HD + (key & 15) * HD + gc * 8;
      __builtin_amdgcn_global_load_lds((const void*)src, MOA_LDS(vs + f * 1024), 16, 0, 0);
    }
  };
  // Transposed V reads (ds_read_b64_tr_b16: within each 16 lanes, lane 4b+e
  // receives element e of the 8-byte reads of lanes 4a+b, a = 0..3). Lane
  // 4a+b of group g reads row 16u + 4(l/32) + a (+8), dims
  // 32d + 16(g%2) + 4b .. +4; after the transpose lane l holds dim 32d + l%32
  // of rows 16u + 4(l/32) + 0..3 (+8): the A operand of O^T = V^T P^T with the
  // slot order of P below.
  const int ta = (lane & 15) >> 2, tb = lane & 3, tg = lane >> 4;
  unsigned vcol[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d)
    vcol[d] = (unsigned)((((4 * d + 2 * (tg & 1) + (tb >> 1)) ^ (2 * ta)) * 16) + 8 * (tb & 1));
  const unsigned vrowoff = (unsigned)((4 * hf + ta) * ROWB);
  auto barrier = [] {
    wait_lgkm0();
    asm volatile("s_barrier" ::: "memory");
  };

  f32x16_t O[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d) O[d] = f32x16_t{};
  float m = -INFINITY, l = 0.f;

  // Every iteration issues the same loads, past the last tile too (keys are
  // clamped to kmax - 1, so those read valid memory and land in slots nobody
  // reads): the number of loads in flight is then the same at every point of
  // the loop, and each wait below is exact rather than a full drain.
  issue_kv(0);
  issue_kv(1);
  for (int t = 0; t < ntile; ++t) {
    // tile t landed (loads issued after it: tile t+1's)
    wait_vmcnt<KPW + VPW>();
    barrier();                               // tile t visible; slots of t-1 free
    issue_kv(t + 2);
    const unsigned char* sl = (sKd + (t % NKS) * KFR * 1024) + lane * 16;
    // two independent accumulation chains (q hi, q lo) keep the MFMA pipe busy
    f32x16_t S = f32x16_t{}, S2 = f32x16_t{};
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      const u32x4 ka = *(const u32x4*)(sl + s * 1024);
      S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, ka), __builtin_bit_cast(bf16x8_t, qh[s]), S, 0, 0, 0);
      S2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, ka), __builtin_bit_cast(bf16x8_t, ql[s]), S2, 0, 0, 0);
    }
    S += S2;
    // causal mask (only tiles that reach past the wave's first query or past
    // kmax need it) and online softmax for query qpos (element e: key kb +
    // 8(e/4) + e%4)
    const int kb = t * TK + 4 * hf;
    if (t * TK + TK - 1 > it.pos0 + 32 * w || t * TK + TK > kmax) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = kb + 8 * (e >> 2) + (e & 3);
        if (key > qpos || key >= kmax) S[e] = -INFINITY;
      }
    }
    float mx = S[0];
#pragma unroll
    for (int e = 1; e < 16; ++e) mx = fmaxf(mx, S[e]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    // The reference maximum moves only when a score exceeds it by more than
    // 2^8 (log2 units): probabilities then stay below 256, exact in the split
    // and harmless in fp32, and the rescale of O below is rare.
    const float mn = (mx > m + 8.f) ? mx : m;
    const float base = (mn == -INFINITY) ? 0.f : mn;   // a row with no key yet keeps m = -inf
    const float alpha = __builtin_amdgcn_exp2f(m - base);
    float ts = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      S[e] = __builtin_amdgcn_exp2f(S[e] - base);
      ts += S[e];
    }
    ts += __shfl_xor(ts, 32, 64);
    l = l * alpha + ts;
    m = mn;
    if (!__all(alpha == 1.f)) {                // no row's maximum moved: nothing to rescale
#pragma unroll
      for (int d = 0; d < DT; ++d) O[d] *= alpha;
    }
    // O^T += V^T P^T over two 16-key steps; slot j of step u is key 16u + 8(j/4) + 4(l/32) + j%4
    // The V reads are explicit LDS instructions with an explicit wait tied to
    // their registers: the compiler, which cannot tell them from the ring
    // slots the direct loads are filling, would otherwise wait for every load
    // in flight (the tile two ahead included) before the first of them.
    const unsigned vb = lds_addr(sV + (t % NKS) * VFR * 1024) + vrowoff;
    u32x4 va[2][DT];
#pragma unroll
    for (int d = 0; d < DT; ++d) {
      va[0][d] = ds_read_tr16_pair<0 * ROWB, 8 * ROWB>(vb + vcol[d]);
      va[1][d] = ds_read_tr16_pair<16 * ROWB, 24 * ROWB>(vb + vcol[d]);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int d = 0; d < DT; ++d) lgkm_wait_for(va[u][d]);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      unsigned ph[4], pl[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) split_pair(S[8 * u + 2 * j], S[8 * u + 2 * j + 1], ph[j], pl[j]);
      const u32x4 pa = u32x4{ph[0], ph[1], ph[2], ph[3]}, pb = u32x4{pl[0], pl[1], pl[2], pl[3]};
#pragma unroll
      for (int d = 0; d < DT; ++d) {
        O[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, va[u][d]), __builtin_bit_cast(bf16x8_t, pa), O[d], 0, 0, 0);
        O[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, va[u][d]), __builtin_bit_cast(bf16x8_t, pb), O[d], 0, 0, 0);
      }
    }
  }
  wait_vmcnt<0>();                           // no load may land in LDS after this workgroup ends
  // normalise and store: element e of O[d] is dim 32d + 8(e/4) + 4(l/32) + e%4 of row 32w + l%32
  const int r = 32 * w + c32;
  if (r < it.nq) {
    const float inv = 1.f / l;
    const size_t o = ((size_t)(it.row0 + r) * n_h + h) * HD + 4 * hf;
#pragma unroll
    for (int d = 0; d < DT; ++d)
#pragma unroll
      for (int e = 0; e < 16; ++e) store_split(out, out_lo, o + 32 * d + 8 * (e >> 2) + (e & 3), O[d][e] * inv);
  }
}

// Combine the key-range partials of one row (fixed order over ranges).
template <bool BF>
__global__ __launch_bounds__(256) void k_attn_reduce(const ReduceItem* __restrict__ red, const float* __restrict__ pacc,
                                                     const float* __restrict__ pml, void* __restrict__ outv,
                                                     size_t out_lo, int n_h, int hd) {
  // One workgroup per (row, head); G = 256 / hd groups of hd lanes take every
  // G-th slot in one pass, each with its own running maximum (its sums are
  // rescaled when a slot's maximum exceeds it), so no pass over the slots
  // waits for another; then the G groups are merged in fixed order.
  __shared__ float sm[4], sl[4];
  __shared__ float so[256];
  const ReduceItem it = red[blockIdx.y];
  const int h = blockIdx.x;
  const int G = 256 / hd;
  const int g = threadIdx.x / hd, dd = threadIdx.x % hd;
  float M = -INFINITY, L = 0.f, o = 0.f;
#pragma unroll 4
  for (int s = g; s < it.nslots; s += G) {
    const size_t b = (size_t)(it.slot0 + s) * n_h + h;
    const float ms = pml[b * 2], ls = pml[b * 2 + 1], as = pacc[b * hd + dd];
    const float mn = fmaxf(M, ms);
    const float wa = __builtin_amdgcn_exp2f(M - mn), wb = __builtin_amdgcn_exp2f(ms - mn);
    L = L * wa + ls * wb;
    o = o * wa + as * wb;
    M = mn;
  }
  so[threadIdx.x] = o;
  if (dd == 0) { sm[g] = M; sl[g] = L; }
  __syncthreads();
  if (g == 0) {
    float Mt = sm[0];
    for (int k = 1; k < G; ++k) Mt = fmaxf(Mt, sm[k]);
    float Lt = 0.f, ot = 0.f;
    for (int k = 0; k < G; ++k) {
      const float w = __builtin_amdgcn_exp2f(sm[k] - Mt);   // a group without slots: -inf -> 0
      Lt += sl[k] * w;
      ot += so[k * hd + dd] * w;
    }
    const size_t oo = ((size_t)it.row * n_h + h) * hd + dd;
    if (BF) store_split((uint16_t*)outv, out_lo, oo, ot / Lt);
    else ((float*)outv)[oo] = ot / Lt;
  }
}

// ------------------------------------------------------------------ argmax
// Greedy sampler: the largest fp32 logit, ties to the lowest token id; the
// token is written into the device token store (it feeds the next step).
__global__ __launch_bounds__(1024) void k_argmax(const float* __restrict__ logits, int V,
                                                 const int* __restrict__ lm_dst, int* __restrict__ tok) {
  __shared__ float sv[16];
  __shared__ int si[16];
  const int r = blockIdx.x;
  const float* lr = logits + (size_t)r * V;
  float best = -INFINITY;
  int bi = INT_MAX;
  // V % 4 == 0: each thread scans float4 groups in increasing index order, so a
  // strict '>' keeps the lowest index among its equal maxima.
  // Eight groups' loads are issued before any of them is compared.
  constexpr int B = 8;
  for (int v0 = threadIdx.x; v0 < V / 4; v0 += 1024 * B) {
    float4 xs[B];
#pragma unroll
    for (int k = 0; k < B; ++k) {
      const int v4 = v0 + 1024 * k;
      xs[k] = (v4 < V / 4) ? *(const float4*)(lr + 4 * v4) : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
    }
#pragma unroll
    for (int k = 0; k < B; ++k) {
      const int v4 = v0 + 1024 * k;
      const float4 x = xs[k];
      if (x.x > best) { best = x.x; bi = 4 * v4; }
      if (x.y > best) { best = x.y; bi = 4 * v4 + 1; }
      if (x.z > best) { best = x.z; bi = 4 * v4 + 2; }
      if (x.w > best) { best = x.w; bi = 4 * v4 + 3; }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ob = __shfl_xor(best, o, 64);
    const int oi = __shfl_xor(bi, o, 64);
    if (ob > best || (ob == best && oi < bi)) { best = ob; bi = oi; }
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) { sv[w] = best; si[w] = bi; }
  __syncthreads();
  if (threadIdx.x == 0) {
    best = sv[0];
    bi = si[0];
    for (int k = 1; k < 16; ++k)
      if (sv[k] > best || (sv[k] == best && si[k] < bi)) { best = sv[k]; bi = si[k]; }
    tok[lm_dst[r]] = (bi == INT_MAX) ? 0 : bi;
  }
}

// ------------------------------------------------------ injected history
template <typename T>
__global__ __launch_bounds__(256) void k_kv_scatter(const T* __restrict__ src, T* __restrict__ kv,
                                                    const int* __restrict__ blocks, int p0, int n, int layer,
                                                    int kv_sel, int NB, int n_kv, int hd) {
  const size_t e = (size_t)blockIdx.x * 256 + threadIdx.x;
  const size_t per = (size_t)n_kv * hd;
  if (e >= (size_t)n * per) return;
  const int p = p0 + (int)(e / per);
  const int rem = (int)(e % per);
  const int h = rem / hd, d = rem - h * hd;
  const size_t hs = (size_t)2 * kBlock * hd;
  const size_t o = (((size_t)layer * NB + blocks[p >> 4]) * n_kv + h) * hs + (size_t)kv_sel * kBlock * hd +
                   (p & 15) * hd + d;
  kv[o] = src[e];
}

__device__ __forceinline__ uint32_t mix32(uint32_t x) {
  x ^= x >> 16; x *= 0x7feb352du; x ^= x >> 15; x *= 0x846ca68bu; x ^= x >> 16;
  return x;
}

template <bool BF>
__global__ __launch_bounds__(256) void k_kv_fill(void* __restrict__ kvv, const int* __restrict__ blocks, int ctx,
                                                 int NB, int n_kv, int hd, uint32_t tag) {
  // grid.y = layer * 2 + (K|V)
  const int layer = blockIdx.y >> 1, kv_sel = blockIdx.y & 1;
  const size_t e = (size_t)blockIdx.x * 256 + threadIdx.x;
  const size_t per = (size_t)n_kv * hd;
  if (e >= (size_t)ctx * per) return;
  const int p = (int)(e / per);
  const int rem = (int)(e % per);
  const int h = rem / hd, d = rem - h * hd;
  const uint32_t u = mix32(tag * 0x9e3779b9u ^ mix32(((uint32_t)blockIdx.y << 24) ^ (uint32_t)p) ^ (uint32_t)(rem * 0x85ebca6bu));
  const float v = (float)(int)(u >> 8) * (1.0f / 8388608.0f) - 1.0f;
  const size_t hs = (size_t)2 * kBlock * hd;
  const size_t o = (((size_t)layer * NB + blocks[p >> 4]) * n_kv + h) * hs + (size_t)kv_sel * kBlock * hd +
                   (p & 15) * hd + d;
  if (BF) ((uint16_t*)kvv)[o] = f2bf(v);
  else ((float*)kvv)[o] = v;
}

// =============================================================== launchers

hipError_t launch_kv_scatter(hipStream_t st, bool bf16, const void* src, void* kv, const int* blocks, int p0, int n,
                             int layer, int kv_sel, int num_blocks, int n_kv, int hd) {
  const size_t total = (size_t)n * n_kv * hd;
  if (total == 0) return hipSuccess;
  const dim3 grid((unsigned)((total + 255) / 256));
  if (bf16)
    klaunch(k_kv_scatter<uint16_t>, grid, dim3(256), st, (const uint16_t*)src, (uint16_t*)kv, blocks, p0, n, layer,
            kv_sel, num_blocks, n_kv, hd);
  else
    klaunch(k_kv_scatter<float>, grid, dim3(256), st, (const float*)src, (float*)kv, blocks, p0, n, layer, kv_sel,
            num_blocks, n_kv, hd);
  return hipGetLastError();
}

hipError_t launch_kv_fill(hipStream_t st, bool bf16, void* kv, const int* blocks, int ctx, int n_layers,
                          int num_blocks, int n_kv, int hd, uint32_t tag) {
  const size_t total = (size_t)ctx * n_kv * hd;
  if (total == 0) return hipSuccess;
  const dim3 grid((unsigned)((total + 255) / 256), 2 * n_layers);
  if (bf16) klaunch(k_kv_fill<true>, grid, dim3(256), st, kv, blocks, ctx, num_blocks, n_kv, hd, tag);
  else klaunch(k_kv_fill<false>, grid, dim3(256), st, kv, blocks, ctx, num_blocks, n_kv, hd, tag);
  return hipGetLastError();
}

hipError_t launch_embed(hipStream_t st, bool bf16, const int* tok_store, const int* row_tok,
                        const int* row_model, ModelPtrs embed, float* x, int T, int d) {
  if (T <= 0) return hipSuccess;
  if (bf16) klaunch(k_embed<true>, dim3(T), dim3(256), st, tok_store, row_tok, row_model, embed, x, d);
  else klaunch(k_embed<false>, dim3(T), dim3(256), st, tok_store, row_tok, row_model, embed, x, d);
  return hipGetLastError();
}

hipError_t launch_add_rmsnorm(hipStream_t st, bool bf16, float* x, const float* part, int nsplit,
                              size_t split_stride, const int* gather, const int* row_model, int nrows,
                              ModelPtrs gamma, void* out, size_t out_lo, int d, float eps) {
  if (nrows <= 0) return hipSuccess;
  if (d % 256 || d > 4096) return hipErrorInvalidValue;
  // V4 float4s per thread (d % 256 == 0: whole waves, at most 1024 threads)
  const int v4 = (d % 2048 == 0) ? 2 : 1;
  const int threads = d / (4 * v4);
  auto go = [&](auto kern) {
    klaunch(kern, dim3(nrows), dim3(threads), st, x, part, nsplit, split_stride, gather, row_model, gamma, out,
            out_lo, d, eps);
  };
  if (bf16) {
    if (v4 == 1) go(k_add_rmsnorm<true, 1>);
    else go(k_add_rmsnorm<true, 2>);
  } else {
    if (v4 == 1) go(k_add_rmsnorm<false, 1>);
    else go(k_add_rmsnorm<false, 2>);
  }
  return hipGetLastError();
}

template <int RT, int CT, int NW, int D, int EPI>
static hipError_t gemm_mm(hipStream_t st, const GemmArgs& a) {
  constexpr unsigned shm = 2 * RT * 1024 * (D + 1);
  static bool attr = false;                           // one attribute call per instantiation
  if (!attr) {
    hipError_t e = hipFuncSetAttribute((const void*)k_gemm_mm<RT, CT, NW, D, EPI>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int nwg = a.total_items;
  klaunch_shm(k_gemm_mm<RT, CT, NW, D, EPI>, dim3((nwg + 7) / 8 * 8), dim3(64 * NW), shm, st, a, nwg);
  return hipGetLastError();
}

// nt: CT (4 waves), 8 + CT (8 waves) or 16 + CT (8 waves, weight ring three
// stages deep); see kMmTile
template <int RT, int EPI>
static hipError_t gemm_mm_nt(hipStream_t st, const GemmArgs& a, int nt) {
  if constexpr (RT <= 4)                          // 4 waves x RT = 8 x CT = 4: one wave per SIMD
    if (nt == 4) return gemm_mm<RT, 4, 4, 3, EPI>(st, a);
  if (nt == 2) return gemm_mm<RT, 2, 4, 4, EPI>(st, a);
  if constexpr (RT >= 4) {
    if (nt == 12) return gemm_mm<RT, 4, 8, (RT >= 8 ? 2 : 3), EPI>(st, a);
    if constexpr (RT >= 8) {
      if (nt == 10 || nt == 18) return gemm_mm<RT, 2, 8, 3, EPI>(st, a);
      if (nt == 20) return gemm_mm<RT, 4, 8, 3, EPI>(st, a);
    }
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gemm(hipStream_t st, bool bf16, const GemmArgs& a, int epi, int mt, int nt) {
  if (a.total_items <= 0) return hipSuccess;
  if (bf16 && mt > kMmTile && mt <= kMmTile + 8) {   // medium-M: 16*RT rows x (16 * NW * CT) columns
    const int rt = mt - kMmTile;
    const int cols = nt > 16 ? 8 * 16 * (nt - 16) : (nt > 8 ? 8 * 16 * (nt - 8) : 4 * 16 * nt);
    if (a.S < 1 || a.S > (a.K >> 5) || a.N % cols != 0) return hipErrorInvalidValue;
    for (int g = 0; g < a.ngroups; ++g)
      if (a.g[g].mrows < 0 || a.g[g].mrows % 16 != 0 || a.g[g].mrows > 16 * rt) return hipErrorInvalidValue;
    if (epi == EPI_SWIGLU) {
      if (rt == 2) return gemm_mm_nt<2, EPI_SWIGLU>(st, a, nt);
      if (rt == 4) return gemm_mm_nt<4, EPI_SWIGLU>(st, a, nt);
      if (rt == 8) return gemm_mm_nt<8, EPI_SWIGLU>(st, a, nt);
    } else {
      if (rt == 2) return gemm_mm_nt<2, EPI_F32>(st, a, nt);
      if (rt == 4) return gemm_mm_nt<4, EPI_F32>(st, a, nt);
      if (rt == 8) return gemm_mm_nt<8, EPI_F32>(st, a, nt);
    }
    return hipErrorInvalidValue;
  }
  if (bf16 && mt >= kWgTile) {
    if (a.ksteps % 4 != 0) return hipErrorInvalidValue;   // the kernel consumes k in stages of 4 steps
    const int m = mt - kWgTile;          // rows / 16
    const int nwg = a.total_items;
    const int grid = (nwg + 7) / 8 * 8;
    const dim3 g(grid), b(256);
#define WGL(M_, N_, E_) klaunch(k_gemm_wg<M_, N_, E_>, g, b, st, a, nwg)
    if (epi == EPI_SWIGLU) {
      if (nt == 4) { if (m == 1) WGL(1, 4, EPI_SWIGLU); else if (m == 2) WGL(2, 4, EPI_SWIGLU); else WGL(4, 4, EPI_SWIGLU); }
      else { if (m == 1) WGL(1, 2, EPI_SWIGLU); else if (m == 2) WGL(2, 2, EPI_SWIGLU); else WGL(4, 2, EPI_SWIGLU); }
    } else {
      if (nt == 4) { if (m == 1) WGL(1, 4, EPI_F32); else if (m == 2) WGL(2, 4, EPI_F32); else WGL(4, 4, EPI_F32); }
      else if (nt == 2) { if (m == 1) WGL(1, 2, EPI_F32); else if (m == 2) WGL(2, 2, EPI_F32); else WGL(4, 2, EPI_F32); }
      else { if (m == 1) WGL(1, 1, EPI_F32); else if (m == 2) WGL(2, 1, EPI_F32); else WGL(4, 1, EPI_F32); }
    }
#undef WGL
    return hipGetLastError();
  }
  if (!bf16) {
    klaunch(k_gemm_f32, dim3(a.total_items), dim3(256), st, a);
    return hipGetLastError();
  }
  return hipErrorInvalidValue;                        // no bf16 kernel for this tile code
}

hipError_t launch_swiglu_f32(hipStream_t st, const float* gu, float* h, int T, int ffn) {
  if (T <= 0) return hipSuccess;
  klaunch(k_swiglu_f32, dim3(T), dim3(256), st, gu, h, ffn);
  return hipGetLastError();
}

hipError_t launch_rope_kv(hipStream_t st, bool bf16, const float* part, int nsplit, size_t split_stride,
                          const int* row_pos, const int* row_bt, const int* bt_store,
                          const float2* rope_tab, float* q, void* kv, int layer, int num_blocks,
                          int n_h, int n_kv, int hd, int T) {
  if (T <= 0) return hipSuccess;
  const int items = (n_h + n_kv) * (hd / 2) + n_kv * hd;
  const dim3 grid(T, (items + 255) / 256);
  if (bf16)
    klaunch(k_rope_kv<true>, grid, dim3(256), st, part, nsplit, split_stride, row_pos, row_bt, bt_store, rope_tab, q, kv,
                                       layer, num_blocks, n_h, n_kv, hd);
  else
    klaunch(k_rope_kv<false>, grid, dim3(256), st, part, nsplit, split_stride, row_pos, row_bt, bt_store, rope_tab, q, kv,
                                        layer, num_blocks, n_h, n_kv, hd);
  return hipGetLastError();
}

#ifndef ATTN_TK64
#define ATTN_TK64 64
#endif
template <int HD, bool BF, int TK = (HD == 64 && BF) ? ATTN_TK64 : 64>
static hipError_t attn_gq(hipStream_t st, int gq, dim3 grid, unsigned shm, const AttnItem* items, const float* q,
                          const void* kv, const int* bt, const int* row_bt, int layer, int NB, int n_h, int n_kv,
                          float sl2, void* out, size_t out_lo, float* pacc, float* pml) {
  switch (gq) {
    case 1: klaunch_shm(k_attn<HD, 1, BF, TK>, grid, dim3(64), shm, st, items, q, kv, bt, row_bt, layer, NB, n_h, n_kv, sl2, out, out_lo, pacc, pml); break;
    case 2: klaunch_shm(k_attn<HD, 2, BF, TK>, grid, dim3(128), shm, st, items, q, kv, bt, row_bt, layer, NB, n_h, n_kv, sl2, out, out_lo, pacc, pml); break;
    case 4: klaunch_shm(k_attn<HD, 4, BF, TK>, grid, dim3(256), shm, st, items, q, kv, bt, row_bt, layer, NB, n_h, n_kv, sl2, out, out_lo, pacc, pml); break;
    case 8: klaunch_shm(k_attn<HD, 8, BF, TK>, grid, dim3(512), shm, st, items, q, kv, bt, row_bt, layer, NB, n_h, n_kv, sl2, out, out_lo, pacc, pml); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attention(hipStream_t st, bool bf16, const AttnItem* items, int nitems, int max_item_blocks,
                            const float* q, const void* kv, const int* bt_store, const int* row_bt,
                            int layer, int num_blocks, int n_h, int n_kv, int hd, float scale,
                            void* out, size_t out_lo, float* pacc, float* pml) {
  if (nitems <= 0) return hipSuccess;

  const unsigned shm = (unsigned)max_item_blocks * 8u;   // one 64-bit block offset per block of an item
  if (shm > 48u * 1024u) return hipErrorInvalidValue;
  const int gq = n_h / n_kv;
  const float sl2 = scale * 1.4426950408889634f;
  dim3 grid(nitems, n_kv);
  if (hd == 64) {
    return bf16 ? attn_gq<64, true>(st, gq, grid, shm, items, q, kv, bt_store, row_bt, layer, num_blocks, n_h, n_kv, sl2, out, out_lo, pacc, pml)
                : attn_gq<64, false>(st, gq, grid, shm, items, q, kv, bt_store, row_bt, layer, num_blocks, n_h, n_kv, sl2, out, out_lo, pacc, pml);
  }
  if (hd == 128) {
    return bf16 ? attn_gq<128, true>(st, gq, grid, shm, items, q, kv, bt_store, row_bt, layer, num_blocks, n_h, n_kv, sl2, out, out_lo, pacc, pml)
                : attn_gq<128, false>(st, gq, grid, shm, items, q, kv, bt_store, row_bt, layer, num_blocks, n_h, n_kv, sl2, out, out_lo, pacc, pml);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_prefill_attention(hipStream_t st, const PrefillItem* items, int nitems, int max_keys,
                                   const float* q, const void* kv, const int* bt_store, int layer, int num_blocks,
                                   int n_h, int n_kv, int hd, float scale, void* out, size_t out_lo) {
  if (nitems <= 0) return hipSuccess;
  // K ring (3 stages of hd/16 1 KB fragments), V ring (3 tiles of 32 rows of
  // hd values), the block ids of the longest item
  const unsigned shm = 3u * (unsigned)(hd / 16) * 1024u + 3u * 32u * (unsigned)hd * 2u +
                       (unsigned)((max_keys + kBlock - 1) / kBlock) * 4u;
  if (max_keys < 1 || shm > kPrefillLdsMax) return hipErrorInvalidValue;
  const dim3 grid(nitems, n_h), blk(256);
  const float sl2 = scale * 1.4426950408889634f;
  static bool attr = false;                // one attribute call per process for both instantiations
  if (!attr) {
    for (const void* f : {(const void*)k_prefill_attn<64>, (const void*)k_prefill_attn<128>}) {
      hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kPrefillLdsMax);
      if (e != hipSuccess) return e;
    }
    attr = true;
  }
  if (hd == 64)
    klaunch_shm(k_prefill_attn<64>, grid, blk, shm, st, items, q, (const uint16_t*)kv, bt_store, layer, num_blocks,
                n_h, n_kv, sl2, (uint16_t*)out, out_lo);
  else if (hd == 128)
    klaunch_shm(k_prefill_attn<128>, grid, blk, shm, st, items, q, (const uint16_t*)kv, bt_store, layer, num_blocks,
                n_h, n_kv, sl2, (uint16_t*)out, out_lo);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attn_reduce(hipStream_t st, bool bf16, const ReduceItem* red, int nred,
                              const float* pacc, const float* pml, void* out, size_t out_lo, int n_h,
                              int hd) {
  if (nred <= 0) return hipSuccess;
  if (hd < 64 || hd > 256 || 256 % hd || nred > 65535) return hipErrorInvalidValue;
  dim3 grid(n_h, nred);                    // heads fastest: a row's heads start together
  if (bf16) klaunch(k_attn_reduce<true>, grid, dim3(256), st, red, pacc, pml, out, out_lo, n_h, hd);
  else klaunch(k_attn_reduce<false>, grid, dim3(256), st, red, pacc, pml, out, out_lo, n_h, hd);
  return hipGetLastError();
}

hipError_t launch_argmax(hipStream_t st, const float* logits, int R, int V, const int* lm_dst, int* tok_store) {
  if (R <= 0) return hipSuccess;
  if (V % 4) return hipErrorInvalidValue;
  klaunch(k_argmax, dim3(R), dim3(1024), st, logits, V, lm_dst, tok_store);
  return hipGetLastError();
}

}  // namespace moa
