// Persistent decode pass for a single episode: every decoder layer of one
// single-token pass (Sec. IV, autoregressive action decode) in one
// cooperative launch of one workgroup per compute unit.
//
// A pass at batch 1 streams all decoder weights once and does almost no
// arithmetic, so its time is set by how continuously HBM is kept busy.  As
// separate launches, each step of a layer pays a launch gap, a ramp-up and a
// tail.  Here the weights never wait for the data: each compute wave streams
// its share of every matrix of every layer, in order, into a ring of 16
// one-KiB fragments in LDS with direct global->LDS loads, and the ring keeps
// running across the grid-wide barriers that separate the steps.  Only the
// multiply waits for the activation vector.  The weight loads are marked
// non-temporal, so the streamed weights do not push the data the workgroups
// exchange, or the keys and values, out of L2.
//
// Steps of a layer (one grid barrier after each):
//  1. QKV projection of RMSNorm(x); the raw q, k, v are published.
//  2. Attention + output projection: the workgroups of head h (one per
//     slice of the output rows, all on one XCD) each compute the head's
//     attention over the cache (the new key and value from the raw q, k, v
//     with RoPE) and multiply it by their slice of W_o's head-h columns,
//     adding the result into an accumulator with device-scope atomic adds.
//     This takes the attention output's round trip through memory and one
//     barrier off the critical path.  The accumulator is a 64-bit integer
//     per output in units of 2^-32: integer addition is associative, so the
//     sum of the head contributions does not depend on the order in which
//     the atomics land and the pass is bit-reproducible.  Quantising a
//     contribution to 2^-32 changes it by at most 2^-33, far below the fp32
//     rounding of the residual; a contribution that is not finite or
//     reaches 2^24 in magnitude sets a poison word instead, and the residual
//     then reads as NaN (the gate fires on a NaN margin).
//  3. Gate/up projection of RMSNorm(r), r = x + accumulator, and SwiGLU;
//     the activation is published.
//  4. Down projection; x = r + result; the accumulator is cleared.
//
// Workgroup layout: 8 compute waves and 1 synchronising wave.
//  * Compute waves stage each step's input into LDS (with the RMSNorm
//    applied), split each block's k range 8 ways (the output projection:
//    its blocks), multiply on MFMA and leave one partial sum per output per
//    wave in LDS.
//  * The synchronising wave sums the partials in a fixed order, applies the
//    epilogue, publishes the results and runs the grid barrier.  It issues no
//    weight loads, so its stores and barrier loads never queue behind the
//    ring in the in-order memory counter.
//  * Data crossing workgroups is written and read with device-coherent (sc1)
//    buffer accesses; the barrier and the accumulator adds use device-scope
//    atomics.  No cache write-back or invalidation is needed.
//
// Work split over the G workgroups (weights as 16-row blocks, see
// gvc_kernels.h): QKV blocks [i*3d/16/G, (i+1)*3d/16/G); down projection
// block i; gate/up pairs [i*F/16/G, (i+1)*F/16/G); step 2: head i % H,
// output slice i / H of min(G/H, d/16) slices.
#include <type_traits>

#include "gvc_kernels.h"

namespace gvc {

namespace {

constexpr int kWaves = 8;                      // compute waves
constexpr int kThreads = (kWaves + 1) * 64;    // plus the synchronising wave
// Weight fragments in flight per compute wave.  Measured on the 7B pass
// (µs per pass): 4: 2862, 6: 2844, 8: 2790, 10: 2799, 11: 2807, 12: 2786,
// 13: 2804, 14: 2816, 16: 2857.
constexpr int kRing = 12;
constexpr int kSC1 = 16;                       // buffer cache policy: device-coherent access
constexpr int kSC0 = 1;                        // buffer cache policy: coherent within an XCD
constexpr int kRingBytes = kWaves * kRing * 1024;
constexpr int kRedBytes = kWaves * kDecodeMaxSeg * 16 * 4;
constexpr int kScoreOffset = 256;              // attention scores follow the head output in the act region
// ring fragments consumed per round in each step (see run_step)
constexpr std::integral_constant<int, 1> kUnQkv{}, kUnGu{}, kUnDown{};
constexpr std::integral_constant<int, 2> kUnO{};

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;

template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }
// Block barrier without a memory fence.  __syncthreads() would also make
// every wave wait for all of its outstanding global loads, the weight ring's
// prefetches of the next step included, before it arrives.  Everything the
// pass shares through a block barrier lives in LDS (each wave's LDS
// operations complete before it arrives); global data written by one
// workgroup and read by another passes through grid_sync / head_sync, whose
// caller waits for its own stores and atomics first, and is read with
// coherent loads.
__device__ __forceinline__ void block_sync() {
  wait_lgkm0();
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ rsrc_t rsrc(const void* p, size_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ float ld_f32(rsrc_t r, int off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kSC1));
}
__device__ __forceinline__ u32x4 ld_b128(rsrc_t r, int off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kSC1);
}
// Exchange within one XCD (device-coherent when `xl` is false): stores are
// written through to the XCD's L2, loads with sc0 miss in the CU's L1.
__device__ __forceinline__ float ld_f32_x(rsrc_t r, int off, bool xl) {
  return xl ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kSC0))
            : __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kSC1));
}
__device__ __forceinline__ void st_f32_x(rsrc_t r, int off, float v, bool xl) {
  if (xl)
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, off, 0, kSC0);
  else
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, off, 0, kSC1);
}
__device__ __forceinline__ u16x8 ld_plain_b128(rsrc_t r, int off) {
  return __builtin_bit_cast(u16x8, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ void st_f32(rsrc_t r, int off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, off, 0, kSC1);
}
__device__ __forceinline__ void st_b16(rsrc_t r, int off, bf16 v) {
  __builtin_amdgcn_raw_buffer_store_b16(v, r, off, 0, kSC1);
}
__device__ __forceinline__ unsigned long long ld_u64(rsrc_t r, int off) {
  typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
  const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kSC1);
  return (unsigned long long)v.x | ((unsigned long long)v.y << 32);
}
__device__ __forceinline__ void st_u64(rsrc_t r, int off, unsigned long long v) {
  typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
  __builtin_amdgcn_raw_buffer_store_b64(u32x2{(unsigned)v, (unsigned)(v >> 32)}, r, off, 0, kSC1);
}

// Fixed-point accumulation of the head contributions (step 2).
constexpr float kFixScale = 4294967296.0f;   // accumulator units per 1.0 (2^32)
constexpr float kFixLimit = 16777216.0f;     // contributions must stay below 2^24 in magnitude
// Residual after attention from the layer input and the accumulator; NaN
// once a contribution was poisoned.
__device__ __forceinline__ float res_value(float x, unsigned long long acc, bool poisoned) {
  const double v = (double)x + (double)(long long)acc * (1.0 / 4294967296.0);
  return poisoned ? __builtin_nanf("") : (float)v;
}
__device__ __forceinline__ bool poisoned_now(const unsigned* bar) {
  return __hip_atomic_load(bar + kDecodePoisonWord, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u;
}

#define GP(p) ((const void __attribute__((address_space(1)))*)(p))
#define LP(p) ((void __attribute__((address_space(3)))*)(p))

// Grid barrier number k of this launch (k >= 1), run by the whole
// synchronising wave.  Per-XCD group counters feed one global counter; the
// targets grow with k, so the counters are zeroed once per launch sequence.
// Returns false after a timeout or when another workgroup timed out.
__device__ bool grid_sync(const DecodeArgs& a, unsigned k) {
  wait_vm<0>();   // this wave's coherent stores and atomics have completed
  int ok = 1;
  if ((threadIdx.x & 63) == 0) {
    const unsigned G = gridDim.x, g = blockIdx.x & 7;
    const unsigned ng = G < 8 ? G : 8;
    const unsigned gsz = (G - g + 7) / 8;
    const unsigned kk = a.bar_base + k;
    const unsigned old = __hip_atomic_fetch_add(a.bar + 32 * (1 + g), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old == gsz * kk - 1) __hip_atomic_fetch_add(a.bar, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const long long t0 = wall_clock64();
    while (__hip_atomic_load(a.bar, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < ng * kk) {
      if (__hip_atomic_load(a.bar + kDecodeAbortWord, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ||
          wall_clock64() - t0 > a.timeout_ticks) {
        __hip_atomic_store(a.bar + kDecodeAbortWord, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  return __builtin_amdgcn_readfirstlane(ok) != 0;
}

// Barrier of the n workgroups of head h (number k of this launch), run by
// the synchronising wave; same timeout and abort rules as grid_sync.
__device__ bool head_sync(const DecodeArgs& a, int h, unsigned n, unsigned k) {
  wait_vm<0>();
  int ok = 1;
  if ((threadIdx.x & 63) == 0) {
    unsigned* ctr = a.bar + kDecodeHeadWord + 32 * h;
    const unsigned target = n * (a.hbar_base + k);
    __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const long long t0 = wall_clock64();
    while (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      if (__hip_atomic_load(a.bar + kDecodeAbortWord, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ||
          wall_clock64() - t0 > a.timeout_ticks) {
        __hip_atomic_store(a.bar + kDecodeAbortWord, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  return __builtin_amdgcn_readfirstlane(ok) != 0;
}

// Staging of a step's input into LDS by the compute waves (threads 0..511;
// the synchronising wave only joins the block barrier).  Their coherent
// loads queue behind the ring in the memory counter, but the ring's loads
// have landed during the grid barrier, and one round trip with 512 threads
// beats several with one wave.
//
// act[0..n) = bf16(src * gain / rms(src)), src fp32 [n], n % 4 == 0,
// n <= NCH * 4 * 512; act[n..npad) = 0.  With RES, src is the residual
// after attention: res_value(x, accumulator) with x = src and the
// accumulator acc.
template <bool RES, int NCH>
__device__ __forceinline__ void stage_norm(rsrc_t src, rsrc_t acc, const unsigned* bar, const float* __restrict__ gain,
                                           int n, int npad, float eps, bf16* act, float* wred) {
  const int tid = threadIdx.x;
  const bool cw = tid < kWaves * 64;
  float4 y[NCH];
  float ss = 0.f;
  if (cw) {
    // every load is issued (indices past the end re-read the last chunk, in
    // bounds) before any is used: one memory round trip, not one per chunk
    // (batches of two chunks with RES: 64-bit accumulators take registers)
    float4 v[NCH], g[NCH];
    constexpr int BATCH = RES ? 2 : NCH;
#pragma unroll
    for (int i0 = 0; i0 < NCH; i0 += BATCH) {
      u32x4 ac[RES ? 2 * BATCH : 1];
#pragma unroll
      for (int i = i0; i < i0 + BATCH; ++i) {
        const int c = min(tid + i * kWaves * 64, n / 4 - 1);
        v[i] = __builtin_bit_cast(float4, ld_b128(src, c * 16));
        g[i] = *(const float4*)(gain + c * 4);
        if constexpr (RES) {
          ac[2 * (i - i0)] = ld_b128(acc, c * 32);
          ac[2 * (i - i0) + 1] = ld_b128(acc, c * 32 + 16);
        }
      }
      if constexpr (RES) {
        const bool poisoned = poisoned_now(bar);
        auto u64 = [](unsigned lo, unsigned hi) { return (unsigned long long)lo | ((unsigned long long)hi << 32); };
#pragma unroll
        for (int i = i0; i < i0 + BATCH; ++i) {
          const u32x4 a0 = ac[2 * (i - i0)], a1 = ac[2 * (i - i0) + 1];
          v[i].x = res_value(v[i].x, u64(a0.x, a0.y), poisoned);
          v[i].y = res_value(v[i].y, u64(a0.z, a0.w), poisoned);
          v[i].z = res_value(v[i].z, u64(a1.x, a1.y), poisoned);
          v[i].w = res_value(v[i].w, u64(a1.z, a1.w), poisoned);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      if (tid + i * kWaves * 64 < n / 4) {
        ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
        y[i] = float4{v[i].x * g[i].x, v[i].y * g[i].y, v[i].z * g[i].z, v[i].w * g[i].w};
      }
    }
ss = wave_sum(ss);
    if ((tid & 63) == 0) wred[tid >> 6] = ss;
  }
  block_sync();
  if (cw) {
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) tot += wred[w];
    const float inv = 1.0f / sqrtf(tot / (float)n + eps);
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int c = tid + i * kWaves * 64;
      if (c < n / 4)
        *(u16x4*)(act + c * 4) = u16x4{f2bf(y[i].x * inv), f2bf(y[i].y * inv), f2bf(y[i].z * inv), f2bf(y[i].w * inv)};
    }
    for (int e = n + tid; e < npad; e += kWaves * 64) act[e] = 0;
  }
}

// act[0..n) = src bf16 [n] (n % 8 == 0, n <= 8 * 2048), act[n..npad) = 0.
__device__ __forceinline__ void stage_copy(rsrc_t src, int n, int npad, bf16* act) {
  const int tid = threadIdx.x;
  if (tid >= kWaves * 64) return;
  u32x4 v[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = ld_b128(src, min(tid + i * kWaves * 64, n / 8 - 1) * 16);   // all loads first
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + i * kWaves * 64;
    if (c < n / 8) *(u32x4*)(act + c * 8) = v[i];
  }
  for (int e = n + tid; e < npad; e += kWaves * 64) act[e] = 0;
}

// Sum over the compute waves of the partials of block s (16 outputs),
// in wave order; lane t < 16 gets output t.
__device__ __forceinline__ float sum_partials(const float* red, int s, int t) {
  float v = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) v += red[(w * kDecodeMaxSeg + s) * 16 + t];
  return v;
}

// Attention of head h for the single token at position pos, computed by each
// of the head's workgroups in full (they share the head's cache lines in
// one L2); the output (DH values, bf16) goes to oact in LDS.  The compute
// waves issue their first loads of the cached keys before the first block
// barrier; meanwhile the synchronising wave applies RoPE to the new q and k
// and, when `append`, writes the new key and value into the caches (for
// later passes).  Position pos itself is read from LDS.  A key (value)
// register is reloaded with the next batch's key (value) as soon as it has
// been used, and the first values are loaded right after the scores, so the
// load round trips overlap the arithmetic and the block barriers.
template <int DH>
__device__ __forceinline__ void attn_head(int h, int pos, int d, int kv_pad, bool append, bool xl, bf16* lkc,
                                          bf16* lvc, const float2* rp, rsrc_t r_qkv, float* qs, float* kn, float* vn,
                                          float* wred, float* sc, bf16* oact) {
  const int tid = threadIdx.x, lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool syncw = wv == kWaves;
  constexpr int half = DH / 2;
  constexpr int NT = kWaves * 64;
  constexpr int LPK = DH / 8, KPI = NT / LPK, U = 5;   // score phase: 8 dims per lane, U key rounds per batch
  constexpr int CG = NT / DH, UV = 5;                  // value phase: CG chunk groups per dim, UV chunks per batch
  const int n_keys = pos + 1, nchunk = (n_keys + 7) / 8;
  const int last_cached = max(pos - 1, 0);
  bf16* kbase = lkc + (size_t)h * kv_pad * DH;
  bf16* vbase = lvc + (size_t)h * DH * kv_pad;
  const rsrc_t r_k = rsrc(kbase, (size_t)kv_pad * DH * 2);
  const rsrc_t r_v = rsrc(vbase, (size_t)kv_pad * DH * 2);
  const int sub = tid % LPK, kg = tid / LPK;           // score phase: key slice, key of the round
  const int koff = sub * 16;
  const int dim = tid / CG, cg = tid % CG;             // value phase: dim, chunk group
  const int voff = dim * kv_pad * 2;
  u16x8 kv[U], vv[UV];
  if (!syncw) {
#pragma unroll
    for (int u = 0; u < U; ++u) kv[u] = ld_plain_b128(r_k, koff + min(u * KPI + kg, last_cached) * DH * 2);
  } else {
    // every load first (one round trip), then RoPE and the appends
    constexpr int NH = (half + 63) / 64, NV = (DH + 63) / 64;
    float q0[NH], q1[NH], k0[NH], k1[NH], vr[NV];
#pragma unroll
    for (int n = 0; n < NH; ++n) {
      const int qo = h * DH + min(lane + 64 * n, half - 1);
      q0[n] = ld_f32_x(r_qkv, qo * 4, xl);
      q1[n] = ld_f32_x(r_qkv, (qo + half) * 4, xl);
      k0[n] = ld_f32_x(r_qkv, (d + qo) * 4, xl);
      k1[n] = ld_f32_x(r_qkv, (d + qo + half) * 4, xl);
    }
#pragma unroll
    for (int n = 0; n < NV; ++n) vr[n] = ld_f32_x(r_qkv, (2 * d + h * DH + min(lane + 64 * n, DH - 1)) * 4, xl);
#pragma unroll
    for (int n = 0; n < NH; ++n) {
      const int i = lane + 64 * n;
      if (i < half) {
        const float2 cs = rp[i];
        qs[i] = q0[n] * cs.x - q1[n] * cs.y;
        qs[i + half] = q1[n] * cs.x + q0[n] * cs.y;
        const bf16 ka = f2bf(k0[n] * cs.x - k1[n] * cs.y), kb = f2bf(k1[n] * cs.x + k0[n] * cs.y);
        kn[i] = bf2f(ka);
        kn[i + half] = bf2f(kb);
        if (append) {
          st_b16(r_k, (pos * DH + i) * 2, ka);
          st_b16(r_k, (pos * DH + i + half) * 2, kb);
        }
      }
    }
#pragma unroll
    for (int n = 0; n < NV; ++n) {
      const int i = lane + 64 * n;
      if (i < DH) {
        const bf16 v = f2bf(vr[n]);
        vn[i] = bf2f(v);
        if (append) st_b16(r_v, (i * kv_pad + pos) * 2, v);
      }
    }
  }
  block_sync();
  // scores q . k_j / sqrt(d_h), j <= pos
  float mx = -INFINITY;
  if (!syncw) {
    float qv[8], kv_new[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) { qv[i] = qs[sub * 8 + i]; kv_new[i] = kn[sub * 8 + i]; }
    const float scale = 1.0f / sqrtf((float)DH);
    for (int j0 = 0; j0 < n_keys; j0 += KPI * U) {
      const bool more = j0 + KPI * U < n_keys;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = j0 + u * KPI + kg;
        float s = 0.f;
        if (j == pos) {
#pragma unroll
          for (int i = 0; i < 8; ++i) s += qv[i] * kv_new[i];
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i) s += qv[i] * bf2f(kv[u][i]);
        }
        // the slot takes the next batch's key at once
        if (more) kv[u] = ld_plain_b128(r_k, koff + min(j + KPI * U, last_cached) * DH * 2);
s = group_sum<LPK>(s);
        s *= scale;
        if (j < n_keys) {
          if (sub == 0) sc[j] = s;
          mx = fmaxf(mx, s);
        }
      }
    }
    // the first values are in flight through the softmax
#pragma unroll
    for (int u = 0; u < UV; ++u) vv[u] = ld_plain_b128(r_v, voff + min(cg + CG * u, nchunk - 1) * 16);
    mx = wave_max(mx);
    if (lane == 0) wred[wv] = mx;
  }
  block_sync();
  float sm = 0.f;
  if (!syncw) {
    mx = wred[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) mx = fmaxf(mx, wred[w]);
    for (int j = tid; j < n_keys; j += NT) {
      const float p = __expf(sc[j] - mx);
      sc[j] = p;
      sm += p;
    }
    sm = wave_sum(sm);
  }
  block_sync();
  if (!syncw) {
    if (lane == 0) wred[8 + wv] = sm;
    for (int j = n_keys + tid; j < nchunk * 8; j += NT) sc[j] = 0.f;   // pad the last 8-key chunk
  }
  block_sync();
  if (!syncw) {
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) tot += wred[8 + w];
    const float vnew = vn[dim];
    float acc = 0.f;
    for (int c0 = 0; c0 < nchunk; c0 += CG * UV) {
      const bool more = c0 + CG * UV < nchunk;
#pragma unroll
      for (int u = 0; u < UV; ++u) {
        const int c = c0 + cg + CG * u;
        if (c < nchunk) {
          const float4 p0 = *(const float4*)(sc + c * 8), p1 = *(const float4*)(sc + c * 8 + 4);
          const float pp[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
          for (int e = 0; e < 8; ++e) acc += pp[e] * (c * 8 + e == pos ? vnew : bf2f(vv[u][e]));
        }
        if (more) vv[u] = ld_plain_b128(r_v, voff + min(c + CG * UV, nchunk - 1) * 16);
      }
    }
acc = group_sum<CG>(acc);
    if (cg == 0) oact[dim] = f2bf(acc / tot);
  }
  block_sync();
}

}  // namespace

// NCH: staging chunks of 4 values per compute thread, d <= NCH * 2048.
template <int DH, int NCH>
__global__ __launch_bounds__(kThreads) void k_decode_pass(const DecodeArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  u32x4* ring = reinterpret_cast<u32x4*>(lds);                  // [kWaves][kRing][64]
  bf16* act = reinterpret_cast<bf16*>(lds + kRingBytes);        // staged activation; step 2: head output
  float* sc = reinterpret_cast<float*>(lds + kRingBytes + kScoreOffset);   // step 2: attention scores
  float* red = reinterpret_cast<float*>(lds + kRingBytes + a.act_bytes);   // [kWaves][kDecodeMaxSeg][16]
  __shared__ float qs[DH], kn[DH], vn[DH], wred[16];
  __shared__ float2 rp[DH / 2];
  __shared__ int s_ok;
  __shared__ u32x4 sink[64];   // destination of the cache-warming loads

  const int tid = threadIdx.x, lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool syncw = wv == kWaves;
  const int G = gridDim.x, gi = blockIdx.x;
  const int d = a.d, F = a.F, H = a.H;
  const int nq = d / 16, nf = F / 16;
  constexpr int KH = DH / 32;   // k fragments of one head's columns

  // This workgroup's blocks per step and this wave's part of them.
  const int w8 = syncw ? 0 : wv;
  const int k0d = w8 * a.KBd / kWaves, nkd = (w8 + 1) * a.KBd / kWaves - k0d;
  const int k0f = w8 * a.KBf / kWaves, nkf = (w8 + 1) * a.KBf / kWaves - k0f;
  // head ah, slice asl of nsl: this workgroup's share of steps 1 and 2
  const int nsl = min(G / H, nq);
  const int ah = gi % H, asl = gi / H;
  const bool attn = asl < nsl;
  // step 1: blocks [qb0, qb0 + nbm) of each of q, k, v within head ah's rows (k split)
  constexpr int BH = DH / 16;
  const int qb0 = attn ? ah * BH + asl * BH / nsl : 0, nbm = attn ? (asl + 1) * BH / nsl - asl * BH / nsl : 0;
  const int nseg0 = 3 * nbm;
  const int sb0 = attn ? asl * nq / nsl : 0, nsb = attn ? (asl + 1) * nq / nsl - sb0 : 0;
  const int ob0w = w8 * nsb / kWaves, nseg_o = syncw ? 0 : (w8 + 1) * nsb / kWaves - ob0w;
  const int gp0 = gi * nf / G, nseg2 = 2 * ((gi + 1) * nf / G - gp0);     // gate, up, gate, up, ...
  const int db0 = gi * nq / G, nseg3 = (gi + 1) * nq / G - db0;           // down blocks (k split)
  const int nsegs = nseg0 + nseg_o + nseg2 + nseg3;   // segments of one layer, in stream order
  // step 5 (kDecodeHead): LM head blocks [hb0, hb0 + nh) (k split), streamed
  // as one more "layer" after the last one
  const bool head = (a.flags & kDecodeHead) != 0;
  const int hb0 = head ? gi * a.nlm / G : 0, nh = head ? (gi + 1) * a.nlm / G - hb0 : 0;
  const int Lend = a.L + (head ? 1 : 0);

  const rsrc_t r_x = rsrc(a.x, (size_t)d * 4), r_acc = rsrc(a.racc, (size_t)d * 8);
  const rsrc_t r_qkv = rsrc(a.qkv, (size_t)3 * d * 4);
  const rsrc_t r_act = rsrc(a.act, (size_t)F * 2);

  // First fragment of segment sg of layer 0 for this wave (offset from wq,
  // in bf16x8 units) and its length.  Everything here is wave-uniform and
  // kept in locals: selects between kernel-argument fields would be turned
  // into indexed private memory.
  const bf16x8* const wq = a.wq;
  const long long off_o = a.wo - a.wq, off_g = a.wg - a.wq, off_d = a.wd - a.wq;
  const bf16x8* const lm0 = head ? a.wlm + ((long long)hb0 * a.KBd + k0d) * 64 : wq;   // head block hb0, k step k0d
  const long long qkv_stride = (long long)a.qkv_stride, gu_stride = (long long)a.gu_stride;
  const long long KBd = a.KBd, KBf = a.KBf;
  auto seg_off = [=](int sg) -> long long {
    if (sg < nseg0) {
      const int m = sg / nbm, rb = qb0 + sg - m * nbm;
      return m * qkv_stride + (rb * KBd + k0d) * 64;
    }
    sg -= nseg0;
    if (sg < nseg_o) return off_o + ((sb0 + ob0w + sg) * KBd + ah * KH) * 64;
    sg -= nseg_o;
    if (sg < nseg2) return off_g + (sg & 1) * gu_stride + ((gp0 + (sg >> 1)) * KBd + k0d) * 64;
    sg -= nseg2;
    return off_d + ((db0 + sg) * KBf + k0f) * 64;
  };
  // (arithmetic rather than a select chain, which becomes an indexed table in private memory)
  auto seg_len = [=](int sg) -> int {
    const int in_o = (sg >= nseg0) & (sg < nseg0 + nseg_o), in_d = sg >= nseg0 + nseg_o + nseg2;
    return nkd + in_o * (KH - nkd) + in_d * (nkf - nkd);
  };

  // Producer state of a compute wave: layer, segment, fragments left in the
  // segment, next fragment (layer 0 address plus layer * layer_stride).
  int p_l = 0, p_sg = 0, p_left = 0;
  const bf16x8* p_ptr = nullptr;
  const bf16x8* last = nullptr;
  int slot = 0;
  u32x4* myring = ring + wv * kRing * 64;
  const bool nt_w = (a.flags & kDecodeNtWeights) != 0;
  const bool streams = !syncw && (nseg0 + nseg2 + nh) * nkd + nseg_o * KH + nseg3 * nkf > 0;
  const long long layer_stride = (long long)a.layer_stride;
  // moves to the next non-empty segment at or after (p_l, p_sg); layer
  // a.L (with the head step) holds the LM head blocks
  auto settle = [&]() {
    while (p_l < Lend) {
      const bool hl = p_l == a.L;
      const int len = hl ? (p_sg < nh ? nkd : 0) : (p_sg < nsegs ? seg_len(p_sg) : 0);   // a layer may have no segments
      if (len > 0) {
        p_ptr = hl ? lm0 + p_sg * KBd * 64 : wq + seg_off(p_sg) + p_l * layer_stride;
        p_left = len;
        return;
      }
      if (++p_sg >= (hl ? nh : nsegs)) { p_sg = 0; ++p_l; }
    }
  };
  auto issue = [&](int sl) {
    const bf16x8* ptr = last;   // past the end: re-read the final fragment (in bounds, cached)
    if (p_l < Lend) {
      ptr = p_ptr;
      last = ptr;
      p_ptr += 64;
      if (--p_left == 0) {
        if (++p_sg >= (p_l == a.L ? nh : nsegs)) { p_sg = 0; ++p_l; }
        settle();
      }
    }
    if (nt_w)
      __builtin_amdgcn_global_load_lds(GP(ptr + lane), LP(myring + sl * 64), 16, 0, 2);
    else
      __builtin_amdgcn_global_load_lds(GP(ptr + lane), LP(myring + sl * 64), 16, 0, 0);
  };
  if (streams) {
    settle();
#pragma unroll 1
    for (int f = 0; f < kRing; ++f) issue(f);
  }

  // Compute waves: nseg blocks of nk k steps each over the staged activation
  // (k steps k0.. of act); partial sums to red[wave][block].  Fragments are
  // consumed UN at a time: the UN oldest ring loads have landed, their LDS
  // reads overlap, then their slots are refilled.  A step whose fragments
  // are already in the ring (the output projection after the attention) is
  // bound by this loop, not by HBM.
  auto run_step = [&](auto un, int nseg, int nk, int k0) {
    constexpr int UN = decltype(un)::value;
    const bf16* abase = act + (lane >> 4) * 8;
    const bool row0 = (lane & 15) == 0;
    for (int s = 0; s < nseg; ++s) {
      floatx4 acc = {0.f, 0.f, 0.f, 0.f};
      int j = 0;
      if constexpr (UN > 1) {
        for (; j + UN <= nk; j += UN) {
          wait_vm<kRing - UN>();
          u32x4 wf[UN], xf[UN];
#pragma unroll
          for (int u = 0; u < UN; ++u) {
            const int sl = slot + u < kRing ? slot + u : slot + u - kRing;
            wf[u] = myring[sl * 64 + lane];
            xf[u] = *(const u32x4*)(abase + (k0 + j + u) * 32);
            if (!row0) xf[u] = u32x4{0u, 0u, 0u, 0u};
          }
#pragma unroll
          for (int u = 0; u < UN; ++u)
            acc = mfma16(__builtin_bit_cast(bf16x8, xf[u]), __builtin_bit_cast(bf16x8, wf[u]), acc);
          wait_lgkm0();
#pragma unroll
          for (int u = 0; u < UN; ++u) {
            issue(slot);
            slot = slot + 1 == kRing ? 0 : slot + 1;
          }
        }
      }
      for (; j < nk; ++j) {
        wait_vm<kRing - 1>();
        const u32x4 wf = myring[slot * 64 + lane];
        u32x4 xf = *(const u32x4*)(abase + (k0 + j) * 32);
        if (!row0) xf = u32x4{0u, 0u, 0u, 0u};
        acc = mfma16(__builtin_bit_cast(bf16x8, xf), __builtin_bit_cast(bf16x8, wf), acc);
        wait_lgkm0();
        issue(slot);
        slot = slot + 1 == kRing ? 0 : slot + 1;
      }
      if (lane < 16) red[(wv * kDecodeMaxSeg + s) * 16 + lane] = acc[0];
    }
    if (nk == 0)   // a wave without k steps contributes zeros
      for (int s = lane; s < nseg * 16; s += 64) red[wv * kDecodeMaxSeg * 16 + s] = 0.f;
  };

  // Synchronising wave: grid barrier; every wave then reads the outcome.
  unsigned nbar = 0;
  auto barrier = [&]() -> bool {
    if (syncw) {
      const bool ok = grid_sync(a, ++nbar);
      if (lane == 0) s_ok = ok;
    }
    block_sync();
    return s_ok != 0;
  };

  // Prologue: clear the accumulator for the first layer's step 2 (each
  // workgroup its down-projection outputs); check that this workgroup runs
  // on XCD blockIdx % 8, which makes each head's workgroups share one L2.
  if (syncw) {
    for (int i = lane; i < DH / 2; i += 64) rp[i] = a.rope[(size_t)a.pos * (DH / 2) + i];
    for (int e = db0 * 16 + lane; e < (db0 + nseg3) * 16; e += 64) st_u64(r_acc, e * 8, 0ull);
    if (lane == 0 && (__builtin_amdgcn_s_getreg((31 << 11) | 20) & 0xf) != (unsigned)(gi & 7))
      __hip_atomic_store(a.bar + kDecodeXccWord, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  bool run = barrier();
  const bool xl = H % 8 == 0 &&
                  __hip_atomic_load(a.bar + kDecodeXccWord, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u;
  unsigned nhbar = 0;

  const float* gains = a.gains;
  int layers_done = 0;
  for (int l = 0; l < a.L && run; ++l) {
    bf16* const lkc = a.kc + (size_t)l * a.kv_layer_elems;
    bf16* const lvc = a.vc + (size_t)l * a.kv_layer_elems;
    // ---------------- 1. QKV projection (head ah's rows, published to the head's workgroups)
    stage_norm<false, NCH>(r_x, r_x, a.bar, gains + (size_t)l * 2 * d, d, a.KBd * 32, a.eps, act, wred);
    block_sync();
    if (!syncw) run_step(kUnQkv, nseg0, nkd, k0d);
    if (syncw && attn && (a.flags & kDecodeWarmKv)) {
      // share asl of head ah's cached keys (rows of DH) and values (dims of
      // kv_pad), read once now so that step 2 finds them in this XCD's L2
      const char* kb = reinterpret_cast<const char*>(lkc + (size_t)ah * a.kv_pad * DH);
      const char* vb = reinterpret_cast<const char*>(lvc + (size_t)ah * DH * a.kv_pad);
      const int r0 = asl * a.pos / nsl, r1 = (asl + 1) * a.pos / nsl;
      for (int o = r0 * DH * 2 + lane * 16; o < r1 * DH * 2; o += 1024)
        __builtin_amdgcn_global_load_lds(GP(kb + o), LP(sink), 16, 0, 0);
      for (int dm = asl * DH / nsl; dm < (asl + 1) * DH / nsl; ++dm)
        for (int o = lane * 16; o < a.pos * 2; o += 1024)
          __builtin_amdgcn_global_load_lds(GP(vb + (size_t)dm * a.kv_pad * 2 + o), LP(sink), 16, 0, 0);
    }
    block_sync();
    if (attn) {
      if (syncw) {
        for (int s0 = 0; s0 < nseg0; s0 += 4) {
          const int s = s0 + (lane >> 4), t = lane & 15;
          if (s < nseg0) {
            const int m = s / nbm, rb = qb0 + s - m * nbm;
            st_f32_x(r_qkv, (m * d + rb * 16 + t) * 4, sum_partials(red, s, t), xl);
          }
        }
        const bool ok = head_sync(a, ah, (unsigned)nsl, ++nhbar);
        if (lane == 0) s_ok = ok;
      }
      block_sync();
      if (!s_ok) break;

      // ---------------- 2. attention of head ah, times W_o's slice asl of head-ah columns
      attn_head<DH>(ah, a.pos, d, a.kv_pad, asl == 0, xl, lkc, lvc, rp, r_qkv, qs, kn, vn, wred, sc, act);
      if (!syncw) run_step(kUnO, nseg_o, KH, 0);
      block_sync();
      if (syncw) {
        bool bad = false;
        for (int w = 0; w < kWaves; ++w) {
          const int wb0 = w * nsb / kWaves, wn = (w + 1) * nsb / kWaves - wb0;
          for (int s0 = 0; s0 < wn; s0 += 4) {
            const int s = s0 + (lane >> 4), t = lane & 15;
            if (s < wn) {
              const float cv = red[(w * kDecodeMaxSeg + s) * 16 + t];
              if (fabsf(cv) < kFixLimit)
                __hip_atomic_fetch_add(a.racc + (sb0 + wb0 + s) * 16 + t,
                                       (unsigned long long)__float2ll_rn(cv * kFixScale), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
              else
                bad = true;
            }
          }
        }
        if (bad) __hip_atomic_store(a.bar + kDecodePoisonWord, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    if (!barrier()) break;

    // ---------------- 3. gate/up projection + SwiGLU
    stage_norm<true, NCH>(r_x, r_acc, a.bar, gains + (size_t)l * 2 * d + d, d, a.KBd * 32, a.eps, act, wred);
    block_sync();
    if (!syncw) run_step(kUnGu, nseg2, nkd, k0d);
    block_sync();
    if (syncw) {
      for (int s0 = 0; s0 < nseg2 / 2; s0 += 4) {
        const int pr = s0 + (lane >> 4), t = lane & 15;
        if (pr < nseg2 / 2) {
          const float g = sum_partials(red, 2 * pr, t), u = sum_partials(red, 2 * pr + 1, t);
          st_b16(r_act, ((gp0 + pr) * 16 + t) * 2, f2bf(g / (1.0f + __expf(-g)) * u));
        }
      }
    }
    if (!barrier()) break;

    // ---------------- 4. down projection + residual; the accumulator is
    // cleared for the next layer's step 2 (every workgroup staged r in step 3,
    // before the last barrier)
    stage_copy(r_act, F, a.KBf * 32, act);
    block_sync();
    if (!syncw) run_step(kUnDown, nseg3, nkf, k0f);
    block_sync();
    if (syncw) {
      const bool poisoned = poisoned_now(a.bar);
      for (int s0 = 0; s0 < nseg3; s0 += 4) {
        const int s = s0 + (lane >> 4), t = lane & 15;
        if (s < nseg3) {
          const int e = (db0 + s) * 16 + t;
          const float rv = res_value(ld_f32(r_x, e * 4), ld_u64(r_acc, e * 8), poisoned);
          st_f32(r_x, e * 4, rv + sum_partials(red, s, t));
          st_u64(r_acc, e * 8, 0ull);
        }
      }
    }
    if (!barrier()) break;
    layers_done = l + 1;
  }

  // ---------------- 5. final RMSNorm, LM head, and this pass's greedy token
  // and margin (Eq. 1): each workgroup writes its logits and one partial
  // record (max, sum of exp, top two bins) of them; after a grid barrier
  // workgroup 0 merges the records in workgroup order (the merge is the same
  // on every run) and writes the token and the margin.
  if (head && layers_done == a.L) {
    stage_norm<false, NCH>(r_x, r_x, a.bar, a.final_gain, d, a.KBd * 32, a.eps, act, wred);
    block_sync();
    if (!syncw) run_step(kUnQkv, nh, nkd, k0d);
    block_sync();
    const rsrc_t r_hp = rsrc(a.head_part, (size_t)G * 8 * 4);
    if (syncw) {
      const rsrc_t r_lg = rsrc(a.logits, (size_t)a.V * 4);
      const int lo = a.full_vocab ? 0 : a.bin_lo;
      float mx = -INFINITY, sm = 0.f, v1 = -INFINITY, v2 = -INFINITY;
      int i1 = 0x7fffffff, i2 = 0x7fffffff;
      for (int s0 = 0; s0 < nh; s0 += 4) {
        const int s = s0 + (lane >> 4), t = lane & 15, idx = (hb0 + s) * 16 + t;
        if (s < nh && idx < a.V) {
          const float z = sum_partials(red, s, t);
          st_f32(r_lg, idx * 4, z);
          if (idx >= lo) lse_add(mx, sm, z);
          if (idx >= a.bin_lo) top2_add(v1, i1, v2, i2, z, idx);
        }
      }
#pragma unroll
      for (int m = 1; m < 64; m <<= 1) {
        lse_merge(mx, sm, __shfl_xor(mx, m), __shfl_xor(sm, m));
        const float w1 = __shfl_xor(v1, m), w2 = __shfl_xor(v2, m);
        const int j1 = __shfl_xor(i1, m), j2 = __shfl_xor(i2, m);
        top2_add(v1, i1, v2, i2, w1, j1);
        top2_add(v1, i1, v2, i2, w2, j2);
      }
      if (lane < 6) {
        const float rec[6] = {mx, sm, v1, __int_as_float(i1), v2, __int_as_float(i2)};
        st_f32(r_hp, (gi * 8 + lane) * 4, rec[lane]);
      }
    }
    if (barrier() && gi == 0 && syncw) {
      float mx = -INFINITY, sm = 0.f, v1 = -INFINITY, v2 = -INFINITY;
      int i1 = 0x7fffffff, i2 = 0x7fffffff;
      for (int w = lane; w < G; w += 64) {
        lse_merge(mx, sm, ld_f32(r_hp, (w * 8) * 4), ld_f32(r_hp, (w * 8 + 1) * 4));
        top2_add(v1, i1, v2, i2, ld_f32(r_hp, (w * 8 + 2) * 4), __float_as_int(ld_f32(r_hp, (w * 8 + 3) * 4)));
        top2_add(v1, i1, v2, i2, ld_f32(r_hp, (w * 8 + 4) * 4), __float_as_int(ld_f32(r_hp, (w * 8 + 5) * 4)));
      }
#pragma unroll
      for (int m = 1; m < 64; m <<= 1) {
        lse_merge(mx, sm, __shfl_xor(mx, m), __shfl_xor(sm, m));
        const float w1 = __shfl_xor(v1, m), w2 = __shfl_xor(v2, m);
        const int j1 = __shfl_xor(i1, m), j2 = __shfl_xor(i2, m);
        top2_add(v1, i1, v2, i2, w1, j1);
        top2_add(v1, i1, v2, i2, w2, j2);
      }
      if (lane == 0) {
        *a.tok_out = i1;
        *a.margin_out = (__expf(v1 - mx) - __expf(v2 - mx)) / sm;
      }
    }
  }
  wait_vm<0>();   // direct-to-LDS loads must land before the workgroup ends
}

size_t decode_pass_lds_bytes(int act_bytes) { return (size_t)kRingBytes + act_bytes + kRedBytes; }

int decode_pass_threads() { return kThreads; }

int decode_pass_score_offset() { return kScoreOffset; }

// d <= 4096: two staging chunks per compute thread (a 4-chunk variant for
// d <= 8192 would spill registers around the 64-bit accumulator loads;
// larger models take the per-step launches).
const void* decode_pass_kernel(int head_dim, int d) {
  if (d > 2 * 4 * kWaves * 64) return nullptr;
  if (head_dim == 128) return reinterpret_cast<const void*>(&k_decode_pass<128, 2>);
  if (head_dim == 64) return reinterpret_cast<const void*>(&k_decode_pass<64, 2>);
  return nullptr;
}

hipError_t launch_decode_pass(const DecodeArgs& a, int n_wg, hipStream_t s) {
  const void* f = decode_pass_kernel(a.head_dim, a.d);
  if (!f) return hipErrorInvalidValue;
  DecodeArgs args = a;
  void* params[] = {&args};
  return hipLaunchCooperativeKernel(f, dim3(n_wg), dim3(kThreads), params,
                                    (unsigned)decode_pass_lds_bytes(a.act_bytes), s);
}

}  // namespace gvc
