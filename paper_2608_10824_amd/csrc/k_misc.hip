// Row bookkeeping, normalisation, embedding, logits reduction, the gate and
// the one-time weight packing.
#include "gvc_kernels.h"

namespace gvc {

// ------------------------------------------------------------------ packing
// Canonical bf16 W[N][K] -> 16-row-block fragment layout (see gvc_kernels.h).
__global__ void k_pack(const bf16* __restrict__ src, int N, int K, bf16* __restrict__ dst, int Nblk, int KB) {
  const size_t total = (size_t)Nblk * KB * 64;
  for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(e & 63);
    const size_t fk = e >> 6;
    const int kb = (int)(fk % KB);
    const int blk = (int)(fk / KB);
    const int n = blk * 16 + (lane & 15);
    const int k = kb * 32 + (lane >> 4) * 8;
    u16x8 v = {0, 0, 0, 0, 0, 0, 0, 0};
    if (n < N) {
      const bf16* row = src + (size_t)n * K;
      if ((K & 7) == 0 && k + 8 <= K) {
        v = *(const u16x8*)(row + k);
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = (k + i < K) ? row[k + i] : (bf16)0;
      }
    }
    *(u16x8*)(dst + e * 8) = v;
  }
}

__global__ void k_convert_gain(const bf16* __restrict__ src, float* __restrict__ dst, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = bf2f(src[i]);
}

// (cos, sin) of pos * theta^(-2i/d_h), evaluated in double then rounded.
__global__ void k_rope_table(float2* __restrict__ tab, int kv_pad, int head_dim, float theta) {
  const int half = head_dim / 2;
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= kv_pad * half) return;
  const int pos = e / half, i = e % half;
  const double ang = (double)pos * pow((double)theta, -2.0 * i / head_dim);
  tab[e] = float2{(float)cos(ang), (float)sin(ang)};
}

__global__ void k_fill_u32(uint32_t* p, uint32_t v, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

// Zeroes positions [from, kv_pad) of n_blk caches of one key layout
// ([kv_pad][dh] per block) and one value layout ([dh][kv_pad] per block).
__global__ void k_zero_kv_tail(bf16* __restrict__ k, bf16* __restrict__ v, size_t n_blk, int kv_pad, int dh,
                               int from) {
  const int tail = kv_pad - from;
  const size_t nk = n_blk * (size_t)tail * dh, nv = n_blk * (size_t)dh * tail;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < nk + nv; i += (size_t)gridDim.x * blockDim.x) {
    if (i < nk) {
      const size_t blk = i / ((size_t)tail * dh), r = i % ((size_t)tail * dh);
      k[blk * kv_pad * dh + (size_t)from * dh + r] = 0;
    } else {
      const size_t j = i - nk, row = j / tail, c = j % tail;   // row = block * dh + dim
      v[row * kv_pad + from + c] = 0;
    }
  }
}

// ------------------------------------------------------------------ row lists
// One workgroup per layer.  Row r = b*P + pos of the batched prompt is
// recomputed at layer l unless episode b has a valid cache, a mask is given,
// pos is a visual token (1..N) and mask[b][l][pos-1] is set.  Writes the
// compacted rows in (b, pos) order as three int arrays (idx, ep, pos) of
// stride B*P, the per-layer count, and per-episode counts and offsets.
__global__ __launch_bounds__(1024) void k_build_rows(const uint8_t* __restrict__ mask, const int* __restrict__ valid,
                                                     int B, int L, int N, int P, int* __restrict__ rows,
                                                     int* __restrict__ counts, int* __restrict__ ep_counts,
                                                     int* __restrict__ ep_offsets) {
  __shared__ int warp_sums[16];
  __shared__ int s_base;
  const int l = blockIdx.x;
  const int total = B * P;
  int* r_idx = rows + (size_t)l * 3 * total;
  int* r_ep = r_idx + total;
  int* r_pos = r_ep + total;
  if (threadIdx.x == 0) s_base = 0;
  __syncthreads();
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  for (int c0 = 0; c0 < total; c0 += 1024) {
    const int r = c0 + threadIdx.x;
    int flag = 0, b = 0, pos = 0;
    if (r < total) {
      b = r / P; pos = r % P;
      flag = 1;
      if (mask && valid[b] && pos >= 1 && pos <= N && mask[((size_t)b * L + l) * N + pos - 1]) flag = 0;
    }
    // inclusive scan within the wave
    int x = flag;
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (lane == 63) warp_sums[wv] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
      int acc = 0;
      for (int w = 0; w < 16; ++w) { const int t = warp_sums[w]; warp_sums[w] = acc; acc += t; }
    }
    __syncthreads();
    const int excl = s_base + warp_sums[wv] + x - flag;
    if (r < total) {
      if (pos == 0) ep_offsets[l * B + b] = excl;
      if (flag) { r_idx[excl] = r; r_ep[excl] = b; r_pos[excl] = pos; }
    }
    __syncthreads();
    if (threadIdx.x == 1023) s_base = excl + flag;
    __syncthreads();
  }
  if (threadIdx.x == 0) counts[l] = s_base;
  __syncthreads();
  if (threadIdx.x < B) {
    const int b = threadIdx.x;
    const int next = (b + 1 < B) ? ep_offsets[l * B + b + 1] : s_base;
    ep_counts[l * B + b] = next - ep_offsets[l * B + b];
  }
}

// ------------------------------------------------------------------ embeddings
// Pixel rows of the layer-0 recomputed rows, frag layout, exact integers in
// bf16; non-visual rows and the padding columns are zero.
__global__ void k_im2row(const uint8_t* __restrict__ frame, int views, int img, int patch,
                         const int* __restrict__ idx, const int* __restrict__ pos_arr, int M, int P, int KB,
                         bf16* __restrict__ x) {
  const int chunks = KB * 4;   // 8-element chunks per row
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= M * chunks) return;
  const int m = e / chunks, k0 = (e % chunks) * 8;
  const int pos = pos_arr[m];
  const int N = views * (img / patch) * (img / patch);
  const int pd = patch * patch * 3;
  u16x8 v = {0, 0, 0, 0, 0, 0, 0, 0};
  if (pos >= 1 && pos <= N) {
    const int b = idx[m] / P;
    const int n = pos - 1;
    const int side = img / patch, per_view = side * side;
    const int vw = n / per_view, rc = n % per_view, r = rc / side, c = rc % side;
    const size_t base = (size_t)b * views * img * img * 3 +
                        ((size_t)vw * img * img + (size_t)r * patch * img + (size_t)c * patch) * 3;
    const int row_bytes = patch * 3;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int k = k0 + i;
      if (k < pd) {
        const int pr = k / row_bytes, pc = k % row_bytes;
        v[i] = f2bf((float)frame[base + (size_t)pr * img * 3 + pc]);
      }
    }
  }
  *(u16x8*)(x + frag_off(m, k0, KB)) = v;
}

// Decode input row b: x = E[token], plus the folded-norm input bf16(x * gain)
// (frag layout) and the row's sum of squares (one part).
__global__ __launch_bounds__(256) void k_embed_tokens(const bf16* __restrict__ embed, const int* __restrict__ tokens,
                                                      int tok_stride, int d, int V, float* __restrict__ x,
                                                      const float* __restrict__ gain, bf16* __restrict__ xn, int KB,
                                                      float* __restrict__ ssq) {
  __shared__ float red[4];
  const int b = blockIdx.x;
  const bf16* e = embed + (size_t)min(max(tokens[b * tok_stride], 0), V - 1) * d;   // ids clamped into [0, V)
  float ss = 0.f;
  for (int f = threadIdx.x * 4; f < d; f += 1024) {
    const float4 v = float4{bf2f(e[f]), bf2f(e[f + 1]), bf2f(e[f + 2]), bf2f(e[f + 3])};
    *(float4*)(x + (size_t)b * d + f) = v;
    const float4 g = *(const float4*)(gain + f);
    *(u16x4*)(xn + frag_off(b, f, KB)) = u16x4{f2bf(v.x * g.x), f2bf(v.y * g.y), f2bf(v.z * g.z), f2bf(v.w * g.w)};
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  if (threadIdx.x == 0) ssq[b] = red[0] + red[1] + red[2] + red[3];
}

// ------------------------------------------------------------------ RMSNorm
// x_out (frag layout bf16) = src_row / sqrt(mean(src_row^2) + eps) * gain.
__global__ __launch_bounds__(256) void k_rmsnorm(const float* __restrict__ src, const int* __restrict__ idx, int d,
                                                 const float* __restrict__ gain, float eps, bf16* __restrict__ x,
                                                 int KB) {
  __shared__ float red[4];
  const int m = blockIdx.x;
  const float* row = src + (size_t)(idx ? idx[m] : m) * d;
  // Rows of up to kRowChunks * 2048 values stay in registers with their
  // gains, every load issued before any is used (chunks past the end re-read
  // the last one, in bounds): one memory round trip.  Longer rows are read
  // twice.  The sum of squares runs in the same order either way.
  constexpr int kRowChunks = 4;
  const int t8 = threadIdx.x * 8;
  float ss = 0.f;
  if (d <= kRowChunks * 256 * 8) {
    float4 ra[kRowChunks], rb[kRowChunks], ga[kRowChunks], gb[kRowChunks];
#pragma unroll
    for (int i = 0; i < kRowChunks; ++i) {
      const int c = min(t8 + i * 256 * 8, d - 8);
      ra[i] = *(const float4*)(row + c);
      rb[i] = *(const float4*)(row + c + 4);
      ga[i] = *(const float4*)(gain + c);
      gb[i] = *(const float4*)(gain + c + 4);
    }
#pragma unroll
    for (int i = 0; i < kRowChunks; ++i) {
      if (t8 + i * 256 * 8 < d) {
        const float4 a = ra[i], b = rb[i];
        ss += a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w + b.x * b.x + b.y * b.y + b.z * b.z + b.w * b.w;
      }
    }
    for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    const float inv = 1.0f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)d + eps);
#pragma unroll
    for (int i = 0; i < kRowChunks; ++i) {
      const int c = t8 + i * 256 * 8;
      if (c < d) {
        const float4 a = ra[i], b = rb[i], g0 = ga[i], g1 = gb[i];
        *(u16x8*)(x + frag_off(m, c, KB)) =
            u16x8{f2bf(a.x * inv * g0.x), f2bf(a.y * inv * g0.y), f2bf(a.z * inv * g0.z), f2bf(a.w * inv * g0.w),
                  f2bf(b.x * inv * g1.x), f2bf(b.y * inv * g1.y), f2bf(b.z * inv * g1.z), f2bf(b.w * inv * g1.w)};
      }
    }
    return;
  }
  for (int c = t8; c < d; c += 256 * 8) {
    const float4 a = *(const float4*)(row + c), b = *(const float4*)(row + c + 4);
    ss += a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w + b.x * b.x + b.y * b.y + b.z * b.z + b.w * b.w;
  }
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float inv = 1.0f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)d + eps);
  for (int c = t8; c < d; c += 256 * 8) {
    const float4 a = *(const float4*)(row + c), b = *(const float4*)(row + c + 4);
    const float4 g0 = *(const float4*)(gain + c), g1 = *(const float4*)(gain + c + 4);
    *(u16x8*)(x + frag_off(m, c, KB)) =
        u16x8{f2bf(a.x * inv * g0.x), f2bf(a.y * inv * g0.y), f2bf(a.z * inv * g0.z), f2bf(a.w * inv * g0.w),
              f2bf(b.x * inv * g1.x), f2bf(b.y * inv * g1.y), f2bf(b.z * inv * g1.z), f2bf(b.w * inv * g1.w)};
  }
}

// The same RMSNorm for one block of 16 rows per workgroup (d % 32 == 0,
// d <= 32 * kNormWaves * kNormFrags): wave w takes k fragments w, w + 8, ...;
// lane l holds row l % 16 and k sub-block l / 16 of each (8 values, kept in
// registers between the sum of squares and the scaling), so every store
// writes one whole 1 KiB fragment.  A row's sum of squares runs per lane over
// its fragments in order, then over the four sub-blocks and the waves in a
// fixed order.  Rows past M (the rest of the last block) repeat row M - 1.
constexpr int kNormWaves = 8, kNormFrags = 16;
__global__ __launch_bounds__(kNormWaves * 64) void k_rmsnorm16(const float* __restrict__ src,
                                                               const int* __restrict__ idx, int M, int d,
                                                               const float* __restrict__ gain, float eps,
                                                               bf16* __restrict__ x, int KB) {
  __shared__ float red[kNormWaves][16];
  __shared__ __attribute__((aligned(16))) float gs[32 * kNormWaves * kNormFrags];   // the gains, staged once
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int mb = blockIdx.x, r = lane & 15, sg = lane >> 4;
  const int m = min(mb * 16 + r, M - 1);
  const float* row = src + (size_t)(idx ? idx[m] : m) * d;
  const int nf = d / 32;
  float4 v[kNormFrags][2];
  float ss = 0.f;
  // every load is issued (fragments past the row's end re-read the last one,
  // in bounds) before any is used: one memory round trip, not one per fragment
#pragma unroll
  for (int i = 0; i < kNormFrags; ++i) {
    const int c = min(w + i * kNormWaves, nf - 1) * 32 + sg * 8;
    v[i][0] = *(const float4*)(row + c);
    v[i][1] = *(const float4*)(row + c + 4);
  }
  // the gains go to LDS in the same round trip (read back after the barrier)
#pragma unroll
  for (int i = 0; i < 32 * kNormWaves * kNormFrags / (kNormWaves * 64 * 4); ++i) {
    const int c = threadIdx.x * 4 + i * kNormWaves * 64 * 4;
    const float4 g = *(const float4*)(gain + min(c, d - 4));
    if (c < d) *(float4*)(gs + c) = g;
  }
#pragma unroll
  for (int i = 0; i < kNormFrags; ++i) {
    if (w + i * kNormWaves < nf) {
      const float4 a = v[i][0], b = v[i][1];
      ss += a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w + b.x * b.x + b.y * b.y + b.z * b.z + b.w * b.w;
    }
  }
  ss += __shfl_xor(ss, 16);
  ss += __shfl_xor(ss, 32);
  if (lane < 16) red[w][lane] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int j = 0; j < kNormWaves; ++j) tot += red[j][r];
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
  for (int i = 0; i < kNormFrags; ++i) {
    const int f = w + i * kNormWaves;
    if (f < nf) {
      const int c = f * 32 + sg * 8;
      const float4 a = v[i][0], b = v[i][1];
      const float4 ga = *(const float4*)(gs + c), gb = *(const float4*)(gs + c + 4);
      const u16x8 o = {f2bf(a.x * inv * ga.x), f2bf(a.y * inv * ga.y), f2bf(a.z * inv * ga.z),
                       f2bf(a.w * inv * ga.w), f2bf(b.x * inv * gb.x), f2bf(b.y * inv * gb.y),
                       f2bf(b.z * inv * gb.z), f2bf(b.w * inv * gb.w)};
      *(u16x8*)(x + ((size_t)(mb * KB + f) * 64 + lane) * 8) = o;
    }
  }
}

// LayerNorm of fp32 rows (ViT blocks): (x - mean) / sqrt(var + eps) * gain
// + bias, the variance taken about the mean in a second pass over the row;
// bf16 out in frag layout.  One workgroup of 256 threads per row; d % 8 == 0.
__global__ __launch_bounds__(256) void k_layernorm(const float* __restrict__ src, int d,
                                                   const float* __restrict__ gain, const float* __restrict__ bias,
                                                   float eps, bf16* __restrict__ x, int KB) {
  __shared__ float red[2][4];
  const int m = blockIdx.x;
  const float* row = src + (size_t)m * d;
  float s = 0.f;
  for (int c = threadIdx.x * 8; c < d; c += 256 * 8) {
    const float4 a = *(const float4*)(row + c), b = *(const float4*)(row + c + 4);
    s += a.x + a.y + a.z + a.w + b.x + b.y + b.z + b.w;
  }
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  if ((threadIdx.x & 63) == 0) red[0][threadIdx.x >> 6] = s;
  __syncthreads();
  const float mean = (red[0][0] + red[0][1] + red[0][2] + red[0][3]) / (float)d;
  float ss = 0.f;
  for (int c = threadIdx.x * 8; c < d; c += 256 * 8) {
    const float4 a = *(const float4*)(row + c), b = *(const float4*)(row + c + 4);
    const float v[8] = {a.x - mean, a.y - mean, a.z - mean, a.w - mean, b.x - mean, b.y - mean, b.z - mean,
                        b.w - mean};
#pragma unroll
    for (int i = 0; i < 8; ++i) ss += v[i] * v[i];
  }
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  if ((threadIdx.x & 63) == 0) red[1][threadIdx.x >> 6] = ss;
  __syncthreads();
  const float inv = 1.0f / sqrtf((red[1][0] + red[1][1] + red[1][2] + red[1][3]) / (float)d + eps);
  for (int c = threadIdx.x * 8; c < d; c += 256 * 8) {
    const float4 a = *(const float4*)(row + c), b = *(const float4*)(row + c + 4);
    const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    u16x8 o;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = f2bf((v[i] - mean) * inv * gain[c + i] + bias[c + i]);
    *(u16x8*)(x + frag_off(m, c, KB)) = o;
  }
}

// Projector input rows of the visual tokens recomputed at layer 0: row m of
// the (position-sorted) list with position 1 <= pos <= N takes frag row
// (episode * N + pos - 1) of src; other rows are zero (their embedding comes
// from the token table or the given rows).  One thread per 8-element chunk.
__global__ void k_gather_visual(const bf16* __restrict__ src, const int* __restrict__ idx,
                                const int* __restrict__ pos_arr, int M, int P, int N, int KB,
                                bf16* __restrict__ x) {
  const int chunks = KB * 4;
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= M * chunks) return;
  const int m = e / chunks, k0 = (e % chunks) * 8;
  const int pos = pos_arr[m];
  u16x8 v = {0, 0, 0, 0, 0, 0, 0, 0};
  if (pos >= 1 && pos <= N) v = *(const u16x8*)(src + frag_off((idx[m] / P) * N + pos - 1, k0, KB));
  *(u16x8*)(x + frag_off(m, k0, KB)) = v;
}

// ------------------------------------------------------------------ logits
// One workgroup per head row: greedy bin token (ties to the lower id) and
// margin p1 - p2 with the softmax normaliser over the whole vocabulary (Eq. 1).
constexpr int kReduceThreads = 1024;
constexpr int kReducePer = 8;   // chunks of 4 logits per thread loaded together

// One pass over the row: every thread keeps its own running maximum, sum of
// exponentials and bin top-2 over a strided set of float4 columns; the
// partial results are merged across the wave, then across the 16 waves.
__global__ __launch_bounds__(kReduceThreads) void k_logits_reduce(const float* __restrict__ logits, int V,
                                                                  int bin_lo, int full_vocab, int* __restrict__ tok_out,
                                                                  float* __restrict__ margin_out, int out_stride,
                                                                  int out_col, int rows_per_ep) {
  constexpr int NW = kReduceThreads / 64;
  __shared__ float s_m[NW], s_s[NW], s_v1[NW], s_v2[NW];
  __shared__ int s_i1[NW], s_i2[NW];
  const int r = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const float4* z4 = (const float4*)(logits + (size_t)r * V);
  const int lo = full_vocab ? 0 : bin_lo;
  const float NEG = -INFINITY;
  float mx = NEG, sum = 0.f;
  // running top-2 of the bins under `better` (a total order: value, then
  // lower id), kept as scalars so that nothing goes to private memory
  float v1 = NEG, v2 = NEG;
  int i1 = 0x7fffffff, i2 = 0x7fffffff;
  // each thread takes chunks tid, tid + T, ... in order; the loads of a batch
  // of kReducePer chunks are all issued before any is used (one round trip)
  const int n4 = V / 4;
  for (int c0 = 0; c0 < n4; c0 += kReduceThreads * kReducePer) {
    float4 q[kReducePer];
#pragma unroll
    for (int u = 0; u < kReducePer; ++u) q[u] = z4[min(c0 + u * kReduceThreads + tid, n4 - 1)];
#pragma unroll
    for (int u = 0; u < kReducePer; ++u) {
      const int c = c0 + u * kReduceThreads + tid;
      if (c < n4) {
        const int i = c * 4;
        const float e[4] = {q[u].x, q[u].y, q[u].z, q[u].w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (i + j >= lo) lse_add(mx, sum, e[j]);
          if (i + j >= bin_lo) top2_add(v1, i1, v2, i2, e[j], i + j);
        }
      }
    }
  }
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) {
    lse_merge(mx, sum, __shfl_xor(mx, m), __shfl_xor(sum, m));
    const float w1 = __shfl_xor(v1, m), w2 = __shfl_xor(v2, m);
    const int j1 = __shfl_xor(i1, m), j2 = __shfl_xor(i2, m);
    top2_add(v1, i1, v2, i2, w1, j1);
    top2_add(v1, i1, v2, i2, w2, j2);
  }
  if (lane == 0) {
    s_m[wv] = mx; s_s[wv] = sum;
    s_v1[wv] = v1; s_i1[wv] = i1; s_v2[wv] = v2; s_i2[wv] = i2;
  }
  __syncthreads();
  if (tid == 0) {
    float M = s_m[0], S = s_s[0];
    v1 = s_v1[0]; i1 = s_i1[0]; v2 = s_v2[0]; i2 = s_i2[0];
    for (int w = 1; w < NW; ++w) {
      lse_merge(M, S, s_m[w], s_s[w]);
      top2_add(v1, i1, v2, i2, s_v1[w], s_i1[w]);
      top2_add(v1, i1, v2, i2, s_v2[w], s_i2[w]);
    }
    const float m = (__expf(v1 - M) - __expf(v2 - M)) / S;
    const int o = (r / rows_per_ep) * out_stride + out_col + r % rows_per_ep;
    tok_out[o] = i1;
    margin_out[o] = m;
  }
}

// ------------------------------------------------------------------ gate
struct Force { signed char f[64]; };

// Alg. 1's test on the previous step's margins: m = mean (Eq. 1) or min over
// the D positions; fire = !(m >= theta) unless forced; a fired episode's
// cache becomes invalid.
__global__ void k_gate(const float* __restrict__ margins, int B, int D, float theta, int use_min, Force force,
                       const unsigned* __restrict__ abort_word, int* __restrict__ valid, float* __restrict__ m_out,
                       int* __restrict__ fire_out) {
  const int b = threadIdx.x;
  if (b >= B) return;
  if (abort_word && *abort_word) {   // the decode that produced the margins did not finish
    valid[b] = 0;                    // invalidation is always safe: the next pass is full
    m_out[b] = __builtin_nanf("");
    fire_out[b] = 1;
    return;
  }
  const float* mr = margins + (size_t)b * D;
  float m;
  if (use_min) {
    m = mr[0];
    for (int j = 1; j < D; ++j) m = fminf(m, mr[j]);
    for (int j = 0; j < D; ++j) if (mr[j] != mr[j]) m = mr[j];   // NaN propagates
  } else {
    float s = 0.f;
    for (int j = 0; j < D; ++j) s += mr[j];
    m = s / (float)D;
  }
  int fire = !(m >= theta);
  if (force.f[b] >= 0) fire = force.f[b] > 0;
  if (fire) valid[b] = 0;
  m_out[b] = m;
  fire_out[b] = fire;
}

// ------------------------------------------------------------------ launchers
hipError_t launch_pack(const bf16* src, int N, int K, bf16* dst, int Nblk, int KB, hipStream_t s) {
  const size_t total = (size_t)Nblk * KB * 64;
  const int blocks = (int)std::min<size_t>((total + 255) / 256, 65536);
  hipLaunchKernelGGL(k_pack, dim3(blocks), dim3(256), 0, s, src, N, K, dst, Nblk, KB);
  return hipGetLastError();
}

hipError_t launch_convert_gain(const bf16* src, float* dst, int n, hipStream_t s) {
  hipLaunchKernelGGL(k_convert_gain, dim3((n + 255) / 256), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

hipError_t launch_rope_table(float2* tab, int kv_pad, int head_dim, float theta, hipStream_t s) {
  const int n = kv_pad * head_dim / 2;
  hipLaunchKernelGGL(k_rope_table, dim3((n + 255) / 256), dim3(256), 0, s, tab, kv_pad, head_dim, theta);
  return hipGetLastError();
}

hipError_t launch_fill_u32(uint32_t* p, uint32_t v, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 65536);
  hipLaunchKernelGGL(k_fill_u32, dim3(blocks), dim3(256), 0, s, p, v, n);
  return hipGetLastError();
}

hipError_t launch_zero_kv_tail(bf16* k, bf16* v, size_t n_blk, int kv_pad, int dh, int from, hipStream_t s) {
  if (from >= kv_pad || n_blk == 0) return hipSuccess;
  const size_t n = 2 * n_blk * (size_t)(kv_pad - from) * dh;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 65536);
  hipLaunchKernelGGL(k_zero_kv_tail, dim3(blocks), dim3(256), 0, s, k, v, n_blk, kv_pad, dh, from);
  return hipGetLastError();
}

hipError_t launch_build_rows(const uint8_t* mask, const int* valid, int B, int L, int N, int P, int* rows,
                             int* counts, int* ep_counts, int* ep_offsets, hipStream_t s) {
  hipLaunchKernelGGL(k_build_rows, dim3(L), dim3(1024), 0, s, mask, valid, B, L, N, P, rows, counts, ep_counts,
                     ep_offsets);
  return hipGetLastError();
}

hipError_t launch_im2row(const uint8_t* frame, int views, int img, int patch, const int* idx, const int* pos,
                         int M, int P, int KB, bf16* x, hipStream_t s) {
  const int n = M * KB * 4;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_im2row, dim3((n + 255) / 256), dim3(256), 0, s, frame, views, img, patch, idx, pos, M, P, KB, x);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(const float* src, const int* idx, int M, int d, const float* gain, float eps, bf16* x,
                          int KB, bool tiled, hipStream_t s) {
  if (M == 0) return hipSuccess;
  if (tiled && d % 32 == 0 && d <= 32 * kNormWaves * kNormFrags)
    hipLaunchKernelGGL(k_rmsnorm16, dim3((M + 15) / 16), dim3(kNormWaves * 64), 0, s, src, idx, M, d, gain, eps, x,
                       KB);
  else
    hipLaunchKernelGGL(k_rmsnorm, dim3(M), dim3(256), 0, s, src, idx, d, gain, eps, x, KB);
  return hipGetLastError();
}

hipError_t launch_layernorm(const float* src, int M, int d, const float* gain, const float* bias, float eps,
                            bf16* x, int KB, hipStream_t s) {
  if (M == 0) return hipSuccess;
  if (d % 8) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_layernorm, dim3(M), dim3(256), 0, s, src, d, gain, bias, eps, x, KB);
  return hipGetLastError();
}

hipError_t launch_gather_visual(const bf16* src, const int* idx, const int* pos, int M, int P, int N, int KB,
                                bf16* x, hipStream_t s) {
  const int n = M * KB * 4;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_gather_visual, dim3((n + 255) / 256), dim3(256), 0, s, src, idx, pos, M, P, N, KB, x);
  return hipGetLastError();
}

hipError_t launch_embed_tokens(const bf16* embed, const int* tokens, int tok_stride, int B, int d, int V, float* x,
                               const float* gain, bf16* xn, int KB, float* ssq, hipStream_t s) {
  hipLaunchKernelGGL(k_embed_tokens, dim3(B), dim3(256), 0, s, embed, tokens, tok_stride, d, V, x, gain, xn, KB, ssq);
  return hipGetLastError();
}

hipError_t launch_logits_reduce(const float* logits, int rows, int V, int bin_lo, int full_vocab, int* tok_out,
                                float* margin_out, int out_stride, int out_col, int rows_per_ep, hipStream_t s) {
  hipLaunchKernelGGL(k_logits_reduce, dim3(rows), dim3(kReduceThreads), 0, s, logits, V, bin_lo, full_vocab, tok_out,
                     margin_out, out_stride, out_col, rows_per_ep);
  return hipGetLastError();
}

hipError_t launch_gate(const float* margins, int B, int D, float theta, int use_min, const int8_t* force,
                       const unsigned* abort_word, int* valid, float* m_out, int* fire_out, hipStream_t s) {
  Force f;
  for (int b = 0; b < 64; ++b) f.f[b] = (force && b < B) ? force[b] : -1;
  hipLaunchKernelGGL(k_gate, dim3(1), dim3(64), 0, s, margins, B, D, theta, use_min, f, abort_word, valid, m_out,
                     fire_out);
  return hipGetLastError();
}

}  // namespace gvc
