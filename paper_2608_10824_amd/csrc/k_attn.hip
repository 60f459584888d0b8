// Causal attention of the recomputed query rows over the mixed K/V cache.
//
// Alg. 1's partial forward pass recomputes only some tokens; their queries
// attend over keys of which some were just written (recomputed rows) and the
// rest are carried over from the previous frame (reused rows).  Both sit in
// the same per-layer cache, so the kernel is an ordinary causal attention
// whose queries are an arbitrary, position-sorted subset of the prompt.
//
// Prefill: one wave per (episode, head, 16 query rows).  S = Q K^T and O += P V
// run on MFMA v_mfma_f32_16x16x32_bf16 over key tiles of 32 with an fp32
// online softmax; P is re-laid out through a 1 KiB LDS tile into the A
// operand order; V is stored transposed so the B operand of P V is 16
// contiguous bytes per lane.
// Decode: one workgroup per (head, episode) and one query.
#include "gvc_kernels.h"

namespace gvc {

template <int DH>
__global__ __launch_bounds__(64) void k_attn_prefill(const bf16* __restrict__ q, const bf16* __restrict__ kc,
                                                     const bf16* __restrict__ vc, const int* __restrict__ rows_pos,
                                                     const int* __restrict__ ep_counts,
                                                     const int* __restrict__ ep_offsets, int H, int kv_pad,
                                                     bf16* __restrict__ o, int KB) {
  constexpr int NK = DH / 32;   // k-steps of QK^T
  constexpr int NO = DH / 16;   // output column blocks
  __shared__ bf16 ps[16 * 32];
  const int tile = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int cnt = ep_counts[b];
  if (tile * 16 >= cnt) return;
  const int off = ep_offsets[b];
  const int lane = threadIdx.x;
  const int col = lane & 15, grp = lane >> 4;
  const int d = H * DH;
  const int last = min(cnt, tile * 16 + 16) - 1;     // last valid row of the tile
  const int max_pos = rows_pos[off + last];
  // this lane's rows in the C layout
  int qpos[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = min(tile * 16 + grp * 4 + i, last);
    qpos[i] = rows_pos[off + r];
  }
  // Q fragments (A operand): row col, dims grp*8 + 32*kk
  bf16x8 qf[NK];
  {
    const int r = min(tile * 16 + col, last);
    const bf16* qr = q + (size_t)(off + r) * d + h * DH + grp * 8;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) qf[kk] = *(const bf16x8*)(qr + kk * 32);
  }
  const bf16* kbase = kc + (size_t)(b * H + h) * kv_pad * DH;
  const bf16* vbase = vc + (size_t)(b * H + h) * DH * kv_pad;
  const float scale = 1.0f / sqrtf((float)DH);
  floatx4 acc[NO];
#pragma unroll
  for (int c = 0; c < NO; ++c) acc[c] = floatx4{0, 0, 0, 0};
  float m_run[4], l_run[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) { m_run[i] = -INFINITY; l_run[i] = 0.f; }

  for (int j0 = 0; j0 <= max_pos; j0 += 32) {
    floatx4 s0 = {0, 0, 0, 0}, s1 = {0, 0, 0, 0};
    const bf16* k0 = kbase + (size_t)(j0 + col) * DH + grp * 8;
    const bf16* k1 = k0 + 16 * DH;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      s0 = mfma16(qf[kk], *(const bf16x8*)(k0 + kk * 32), s0);
      s1 = mfma16(qf[kk], *(const bf16x8*)(k1 + kk * 32), s1);
    }
    float p0[4], p1[4], alpha[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float a0 = (j0 + col <= qpos[i]) ? s0[i] * scale : -INFINITY;
      const float a1 = (j0 + 16 + col <= qpos[i]) ? s1[i] * scale : -INFINITY;
      float mx = fmaxf(a0, a1);
      for (int x = 1; x < 16; x <<= 1) mx = fmaxf(mx, __shfl_xor(mx, x));
      const float mn = fmaxf(m_run[i], mx);
      alpha[i] = __expf(m_run[i] - mn);
      p0[i] = __expf(a0 - mn);
      p1[i] = __expf(a1 - mn);
      float sm = p0[i] + p1[i];
      for (int x = 1; x < 16; x <<= 1) sm += __shfl_xor(sm, x);
      l_run[i] = l_run[i] * alpha[i] + sm;
      m_run[i] = mn;
    }
#pragma unroll
    for (int c = 0; c < NO; ++c)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[c][i] *= alpha[i];
    // P (C layout: row grp*4+i, key col / 16+col) -> LDS [16][32] -> A layout
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ps[(grp * 4 + i) * 32 + col] = f2bf(p0[i]);
      ps[(grp * 4 + i) * 32 + 16 + col] = f2bf(p1[i]);
    }
    __syncthreads();
    const bf16x8 pa = *(const bf16x8*)(ps + col * 32 + grp * 8);
    __syncthreads();
    const bf16* vj = vbase + j0 + grp * 8;
#pragma unroll
    for (int c = 0; c < NO; ++c) {
      const bf16x8 vb = *(const bf16x8*)(vj + (size_t)(c * 16 + col) * kv_pad);
      acc[c] = mfma16(pa, vb, acc[c]);
    }
  }
  // normalise and store (frag layout for the output projection)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = tile * 16 + grp * 4 + i;
    if (r >= cnt) continue;
    const int m = off + r;
    const float inv = 1.0f / l_run[i];
#pragma unroll
    for (int c = 0; c < NO; ++c) o[frag_off(m, h * DH + c * 16 + col, KB)] = f2bf(acc[c][i] * inv);
  }
}

// One workgroup per (head, episode): a single query at position n_keys-1.
// Scores: DH/8 lanes per key, each lane a 16-byte run of dims, so one wave
// instruction reads whole key rows contiguously; partial dots are summed
// across the lane group.  Values: the cache is dim-major, so a lane reads
// 8 consecutive keys of one dim and a wave instruction reads 4 dims x 16
// chunks = 4 contiguous 256-byte runs.  Both phases issue a batch of loads
// (clamped addresses, results masked) before consuming any of them, so the
// kernel pays the memory latency a few times rather than once per key group.
template <int DH>
__global__ __launch_bounds__(256) void k_attn_decode(const bf16* __restrict__ q, const bf16* __restrict__ kc,
                                                     const bf16* __restrict__ vc, int H, int kv_pad, int n_keys,
                                                     bf16* __restrict__ o, int KB) {
  extern __shared__ float sc[];          // [kv_pad] scores, then probabilities
  __shared__ float red[8];
  constexpr int LPK = DH / 8;            // lanes per key
  constexpr int KPI = 256 / LPK;         // keys per load round
  constexpr int U = 8;                   // load rounds per batch
  constexpr int ND = DH / 16;            // dims per thread in the value phase
  constexpr int UC = 3;                  // 8-key chunks per lane per value batch
  const int h = blockIdx.x, b = blockIdx.y;
  const int d = H * DH;
  const int tid = threadIdx.x;
  const int sub = tid % LPK, kg = tid / LPK;
  float qv[8];
  {
    const u16x8 qq = *(const u16x8*)(q + (size_t)b * d + h * DH + sub * 8);
#pragma unroll
    for (int i = 0; i < 8; ++i) qv[i] = bf2f(qq[i]);
  }
  const bf16* kbase = kc + (size_t)(b * H + h) * kv_pad * DH + sub * 8;
  const float scale = 1.0f / sqrtf((float)DH);
  float mx = -INFINITY;
  for (int j0 = 0; j0 < n_keys; j0 += KPI * U) {
    u16x8 kv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) kv[u] = *(const u16x8*)(kbase + (size_t)min(j0 + u * KPI + kg, n_keys - 1) * DH);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u * KPI + kg;
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) s += qv[i] * bf2f(kv[u][i]);
#pragma unroll
      for (int x = LPK / 2; x > 0; x >>= 1) s += __shfl_xor(s, x);
      s *= scale;
      if (j < n_keys) {
        if (sub == 0) sc[j] = s;
        mx = fmaxf(mx, s);
      }
    }
  }
  for (int x = 32; x > 0; x >>= 1) mx = fmaxf(mx, __shfl_xor(mx, x));
  if ((tid & 63) == 0) red[tid >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  float sm = 0.f;
  for (int j = tid; j < n_keys; j += 256) {
    const float p = __expf(sc[j] - mx);
    sc[j] = p;
    sm += p;
  }
  for (int x = 32; x > 0; x >>= 1) sm += __shfl_xor(sm, x);
  if ((tid & 63) == 0) red[4 + (tid >> 6)] = sm;
  for (int j = n_keys + tid; j < (n_keys + 7) / 8 * 8; j += 256) sc[j] = 0.f;   // pad the last 8-key chunk
  __syncthreads();
  const float inv = 1.0f / (red[4] + red[5] + red[6] + red[7]);
  // o[dim] = sum_j p_j V^T[dim][j]: lane16 walks 8-key chunks, 16 dim groups
  const int l16 = tid & 15, dg = tid >> 4;
  const int nchunk = (n_keys + 7) / 8;
  const bf16* vb = vc + (size_t)(b * H + h) * DH * kv_pad + (size_t)dg * kv_pad;
  float acc[ND];
#pragma unroll
  for (int i = 0; i < ND; ++i) acc[i] = 0.f;
  for (int c0 = 0; c0 < nchunk; c0 += 16 * UC) {
    u16x8 vv[ND][UC];
#pragma unroll
    for (int i = 0; i < ND; ++i)
#pragma unroll
      for (int u = 0; u < UC; ++u)
        vv[i][u] = *(const u16x8*)(vb + (size_t)(16 * i) * kv_pad + min(c0 + 16 * u + l16, nchunk - 1) * 8);
#pragma unroll
    for (int u = 0; u < UC; ++u) {
      const int c = c0 + 16 * u + l16;
      if (c < nchunk) {
        const float4 p0 = *(const float4*)(sc + c * 8), p1 = *(const float4*)(sc + c * 8 + 4);
        const float pp[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
        for (int i = 0; i < ND; ++i)
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[i] += pp[e] * bf2f(vv[i][u][e]);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < ND; ++i) {
    float t = acc[i];
#pragma unroll
    for (int x = 8; x > 0; x >>= 1) t += __shfl_xor(t, x);
    if (l16 == 0) o[frag_off(b, h * DH + dg + 16 * i, KB)] = f2bf(t * inv);
  }
}

hipError_t launch_attn_prefill(const bf16* q, const bf16* kc, const bf16* vc, const int* rows_pos,
                               const int* ep_counts, const int* ep_offsets, int B, int H, int head_dim, int kv_pad,
                               int max_tiles, bf16* o, int KB, hipStream_t s) {
  dim3 grid(max_tiles, H, B);
  if (head_dim == 128)
    hipLaunchKernelGGL(k_attn_prefill<128>, grid, dim3(64), 0, s, q, kc, vc, rows_pos, ep_counts, ep_offsets, H,
                       kv_pad, o, KB);
  else if (head_dim == 64)
    hipLaunchKernelGGL(k_attn_prefill<64>, grid, dim3(64), 0, s, q, kc, vc, rows_pos, ep_counts, ep_offsets, H,
                       kv_pad, o, KB);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attn_decode(const bf16* q, const bf16* kc, const bf16* vc, int B, int H, int head_dim, int kv_pad,
                              int n_keys, bf16* o, int KB, hipStream_t s) {
  dim3 grid(H, B);
  const size_t shm = (size_t)kv_pad * sizeof(float);
  if (head_dim == 128)
    hipLaunchKernelGGL(k_attn_decode<128>, grid, dim3(256), shm, s, q, kc, vc, H, kv_pad, n_keys, o, KB);
  else if (head_dim == 64)
    hipLaunchKernelGGL(k_attn_decode<64>, grid, dim3(256), shm, s, q, kc, vc, H, kv_pad, n_keys, o, KB);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace gvc
