// Gathered-row GEMM for the projections and the FFN: C[m][n] = X[m][:] . W[n][:].
//
// Each projection of a (partial) prompt pass or of a single-token decode pass
// runs over the M recomputed token rows only (Alg. 1, partial forward pass).
// M is small next to the weight matrices (1 to a few hundred rows per episode),
// so the kernel is built around streaming the packed bf16 weights once:
//  * MFMA v_mfma_f32_16x16x32_bf16 with the weight block as the A operand
//    (16 output features) and 16 token rows as the B operand; every lane loads
//    16 contiguous bytes of both operands straight from their packed layouts;
//  * one wave owns a PAIR of 16-row weight blocks for all the tile's token
//    rows; the pair is chosen so that the epilogue's partner values sit in
//    the same lane and register: RoPE dims (i, i + d_h/2), SwiGLU (gate j, up j);
//  * 4 waves per workgroup share the token fragments through LDS (NT > 1);
//  * weight fragments are prefetched PF k-steps ahead in registers;
//  * split-K across workgroups: partial tiles go to a workspace, the last
//    workgroup of a tile (atomic ticket) sums them in fixed split order, so
//    results are bitwise reproducible, then runs the epilogue.
#include "gvc_kernels.h"

namespace gvc {

__device__ __forceinline__ void map_pair(const GemmArgs& a, int pair, int& mat_a, int& blk_a, int& mat_b,
                                         int& blk_b, bool& b_ok) {
  b_ok = true;
  if (a.map == MAP_QKV) {
    const int dh = a.e.head_dim;
    const int per_mat = a.wblk[0] >> 1;        // pairs per d x d matrix
    const int m = pair / per_mat, pp = pair % per_mat;
    const int per_head = dh >> 5;              // pairs per head
    const int head = pp / per_head, j = pp % per_head;
    mat_a = mat_b = m;
    blk_a = head * (dh >> 4) + j;
    blk_b = blk_a + per_head;
  } else if (a.map == MAP_GU) {
    mat_a = 0; mat_b = 1; blk_a = blk_b = pair;
  } else {
    mat_a = mat_b = 0;
    blk_a = 2 * pair;
    blk_b = 2 * pair + 1;
    if (blk_b >= a.wblk[0]) { blk_b = blk_a; b_ok = false; }
  }
}

__device__ __forceinline__ float silu_f(float g) { return g / (1.0f + __expf(-g)); }

template <int EPI>
__device__ __forceinline__ void epilogue(const GemmArgs& a, int pair, int lane, int m, const floatx4& va,
                                         const floatx4& vb, bool b_ok) {
  const EpiArgs& e = a.e;
  int mat_a, blk_a, mat_b, blk_b; bool bo;
  map_pair(a, pair, mat_a, blk_a, mat_b, blk_b, bo);
  const int sub = (lane >> 4) * 4;   // first of the 4 features this lane holds
  if constexpr (EPI == EPI_QKV) {
    const int dh = e.head_dim, half = dh >> 1;
    const int head = blk_a / (dh >> 4);
    const int ia = (blk_a % (dh >> 4)) * 16 + sub;   // dim within head, < half
    const int pos = e.rows.pos[m];
    const int b = e.rows.ep[m];
    float ra[4], rb[4];
    if (mat_a < 2) {
      const float2* cs = e.rope + (size_t)pos * half + ia;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float2 c = cs[i];
        ra[i] = va[i] * c.x - vb[i] * c.y;
        rb[i] = vb[i] * c.x + va[i] * c.y;
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) { ra[i] = va[i]; rb[i] = vb[i]; }
    }
    if (mat_a == 0) {
      bf16* q = e.q + (size_t)m * e.d + head * dh;
      u16x4 oa = {f2bf(ra[0]), f2bf(ra[1]), f2bf(ra[2]), f2bf(ra[3])};
      u16x4 ob = {f2bf(rb[0]), f2bf(rb[1]), f2bf(rb[2]), f2bf(rb[3])};
      *(u16x4*)(q + ia) = oa;
      *(u16x4*)(q + ia + half) = ob;
    } else if (mat_a == 1) {
      bf16* k = e.kc + ((size_t)(b * e.n_heads + head) * e.kv_pad + pos) * dh;
      u16x4 oa = {f2bf(ra[0]), f2bf(ra[1]), f2bf(ra[2]), f2bf(ra[3])};
      u16x4 ob = {f2bf(rb[0]), f2bf(rb[1]), f2bf(rb[2]), f2bf(rb[3])};
      *(u16x4*)(k + ia) = oa;
      *(u16x4*)(k + ia + half) = ob;
    } else {
      bf16* v = e.vc + (size_t)(b * e.n_heads + head) * dh * e.kv_pad + pos;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[(size_t)(ia + i) * e.kv_pad] = f2bf(ra[i]);
        v[(size_t)(ia + half + i) * e.kv_pad] = f2bf(rb[i]);
      }
    }
  } else if constexpr (EPI == EPI_RESID) {
    const int d = e.d;
    const size_t ri = (size_t)(e.resid_mapped ? e.rows.idx[m] : m) * d;
    const size_t oi = (size_t)(e.out_mapped ? e.rows.idx[m] : m) * d;
    const int fa = blk_a * 16 + sub;
    {
      const float4 r = *(const float4*)(e.resid + ri + fa);
      float4 o; o.x = r.x + va[0]; o.y = r.y + va[1]; o.z = r.z + va[2]; o.w = r.w + va[3];
      *(float4*)(e.out + oi + fa) = o;
    }
    if (b_ok) {
      const int fb = blk_b * 16 + sub;
      const float4 r = *(const float4*)(e.resid + ri + fb);
      float4 o; o.x = r.x + vb[0]; o.y = r.y + vb[1]; o.z = r.z + vb[2]; o.w = r.w + vb[3];
      *(float4*)(e.out + oi + fb) = o;
    }
  } else if constexpr (EPI == EPI_SILU) {
    const int f = blk_a * 16 + sub;
    if (f < e.n_feat) {
      u16x4 o;
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = f2bf(silu_f(va[i]) * vb[i]);
      *(u16x4*)(e.act + frag_off(m, f, e.kb_act)) = o;
    }
  } else if constexpr (EPI == EPI_STORE) {
    float* o = e.store + (size_t)m * e.ld_store;
    const int fa = blk_a * 16 + sub;
    if (fa < a.n_out) *(float4*)(o + fa) = float4{va[0], va[1], va[2], va[3]};
    const int fb = blk_b * 16 + sub;
    if (b_ok && fb < a.n_out) *(float4*)(o + fb) = float4{vb[0], vb[1], vb[2], vb[3]};
  } else {  // EPI_EMBED
    const int d = e.d;
    const int pos = e.rows.pos[m], b = e.rows.ep[m];
    float* h = e.h0 + (size_t)e.rows.idx[m] * d;
    const float inv255 = 1.0f / 255.0f;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      if (half == 1 && !b_ok) break;
      const int f = (half ? blk_b : blk_a) * 16 + sub;
      const floatx4& v = half ? vb : va;
      float4 o;
      if (pos >= 1 && pos <= e.n_patches) {
        o.x = v[0] * inv255; o.y = v[1] * inv255; o.z = v[2] * inv255; o.w = v[3] * inv255;
      } else if (pos < e.n_patches + e.n_text) {
        const int t = pos == 0 ? 0 : pos - e.n_patches;
        const bf16* er = e.embed + (size_t)e.text_ids[b * e.n_text + t] * d + f;
        o.x = bf2f(er[0]); o.y = bf2f(er[1]); o.z = bf2f(er[2]); o.w = bf2f(er[3]);
      } else {
        const float* xr = e.extra + ((size_t)b * e.n_extra + (pos - e.n_patches - e.n_text)) * d + f;
        o = *(const float4*)xr;
      }
      *(float4*)(h + f) = o;
    }
  }
}

template <int NT, int PF, int EPI>
__global__ __launch_bounds__(256) void k_gemm(const GemmArgs a) {
  constexpr int XS = NT > 1 ? NT * PF * 64 : 1;
  __shared__ bf16x8 xs[XS];
  __shared__ int s_last;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int split = blockIdx.x % a.splits, tile = blockIdx.x / a.splits, mt = blockIdx.y;
  const int pair = tile * 4 + wave;
  const bool p_ok = pair < a.n_pairs;
  int mat_a, blk_a, mat_b, blk_b; bool b_ok;
  map_pair(a, p_ok ? pair : 0, mat_a, blk_a, mat_b, blk_b, b_ok);
  const bf16x8* wa = a.w[mat_a] + (size_t)blk_a * a.KB * 64 + lane;
  const bf16x8* wb = a.w[mat_b] + (size_t)blk_b * a.KB * 64 + lane;

  const int kb0 = split * a.kb_per_split;
  const int kb1 = min(a.KB, kb0 + a.kb_per_split);
  const int nsteps = kb1 - kb0;
  const int mb0 = mt * NT;  // first token block of this tile
  const bf16x8* xg = a.x + (size_t)mb0 * a.KB * 64;

  floatx4 acc_a[NT], acc_b[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) { acc_a[t] = floatx4{0, 0, 0, 0}; acc_b[t] = floatx4{0, 0, 0, 0}; }

  bf16x8 ra[PF], rb[PF], rx[NT == 1 ? PF : 1];
  const bf16x8 zero8 = bf16x8{};
#pragma unroll
  for (int p = 0; p < PF; ++p) {
    if (p < nsteps) {
      ra[p] = wa[(size_t)(kb0 + p) * 64];
      rb[p] = wb[(size_t)(kb0 + p) * 64];
      if constexpr (NT == 1) rx[p] = mb0 < a.mblocks ? xg[(size_t)(kb0 + p) * 64 + lane] : zero8;
    }
  }

  for (int base = 0; base < nsteps; base += PF) {
    if constexpr (NT > 1) {
      __syncthreads();
      for (int e = threadIdx.x; e < NT * PF * 64; e += 256) {
        const int t = e / (PF * 64), p = (e >> 6) % PF, ln = e & 63;
        const int kb = kb0 + base + p;
        bf16x8 v = zero8;
        if (kb < kb1 && mb0 + t < a.mblocks) v = xg[((size_t)t * a.KB + kb) * 64 + ln];
        xs[e] = v;
      }
      __syncthreads();
    }
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      const int s = base + p;
      if (s < nsteps) {
        const bf16x8 a0 = ra[p], a1 = rb[p];
        bf16x8 x0 = zero8;
        if constexpr (NT == 1) x0 = rx[p];
        if (s + PF < nsteps) {
          ra[p] = wa[(size_t)(kb0 + s + PF) * 64];
          rb[p] = wb[(size_t)(kb0 + s + PF) * 64];
          if constexpr (NT == 1) rx[p] = mb0 < a.mblocks ? xg[(size_t)(kb0 + s + PF) * 64 + lane] : zero8;
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const bf16x8 xb = NT > 1 ? xs[(t * PF + p) * 64 + lane] : x0;
          acc_a[t] = mfma16(a0, xb, acc_a[t]);
          acc_b[t] = mfma16(a1, xb, acc_b[t]);
        }
      }
    }
  }

  const int col = lane & 15;
  if (a.splits > 1) {
    const int tile_id = tile * a.mtiles + mt;
    floatx4* P = a.part + ((size_t)tile_id * a.splits * 4 + wave) * 2 * NT * 64 + lane;
    const size_t split_stride = (size_t)4 * 2 * NT * 64;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int m = (mb0 + t) * 16 + col;
      if (m < a.M) {
        P[split * split_stride + (size_t)t * 64] = acc_a[t];
        P[split * split_stride + (size_t)(NT + t) * 64] = acc_b[t];
      }
    }
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) s_last = atomicAdd(&a.tickets[tile_id], 1) == a.splits - 1;
    __syncthreads();
    if (!s_last) return;
    __threadfence();
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int m = (mb0 + t) * 16 + col;
      floatx4 sa = floatx4{0, 0, 0, 0}, sb = floatx4{0, 0, 0, 0};
      if (m < a.M) {
        for (int s = 0; s < a.splits; ++s) {
          sa += P[s * split_stride + (size_t)t * 64];
          sb += P[s * split_stride + (size_t)(NT + t) * 64];
        }
      }
      acc_a[t] = sa; acc_b[t] = sb;
    }
    if (threadIdx.x == 0) a.tickets[tile_id] = 0;
  }

  if (!p_ok) return;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int m = (mb0 + t) * 16 + col;
    if (m < a.M) epilogue<EPI>(a, pair, lane, m, acc_a[t], acc_b[t], b_ok);
  }
}

template <int EPI, int NT>
static hipError_t launch_nt(const GemmArgs& a, hipStream_t s) {
  constexpr int PF = NT == 1 ? 8 : (NT <= 8 ? 4 : 2);
  const int tiles = (a.n_pairs + 3) / 4;
  dim3 grid(tiles * a.splits, a.mtiles);
  hipLaunchKernelGGL((k_gemm<NT, PF, EPI>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int EPI>
static hipError_t launch_epi(const GemmArgs& a, int NT, hipStream_t s) {
  switch (NT) {
    case 1: return launch_nt<EPI, 1>(a, s);
    case 2: return launch_nt<EPI, 2>(a, s);
    case 3: return launch_nt<EPI, 3>(a, s);
    case 4: return launch_nt<EPI, 4>(a, s);
    case 5: return launch_nt<EPI, 5>(a, s);
    case 6: return launch_nt<EPI, 6>(a, s);
    case 7: return launch_nt<EPI, 7>(a, s);
    case 8: return launch_nt<EPI, 8>(a, s);
    case 9: return launch_nt<EPI, 9>(a, s);
    case 10: return launch_nt<EPI, 10>(a, s);
    case 11: return launch_nt<EPI, 11>(a, s);
    case 12: return launch_nt<EPI, 12>(a, s);
    case 13: return launch_nt<EPI, 13>(a, s);
    case 14: return launch_nt<EPI, 14>(a, s);
    case 15: return launch_nt<EPI, 15>(a, s);
    case 16: return launch_nt<EPI, 16>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm(const GemmArgs& a, int epi, int NT, hipStream_t s) {
  switch (epi) {
    case EPI_QKV: return launch_epi<EPI_QKV>(a, NT, s);
    case EPI_RESID: return launch_epi<EPI_RESID>(a, NT, s);
    case EPI_SILU: return launch_epi<EPI_SILU>(a, NT, s);
    case EPI_STORE: return launch_epi<EPI_STORE>(a, NT, s);
    case EPI_EMBED: return launch_epi<EPI_EMBED>(a, NT, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace gvc
