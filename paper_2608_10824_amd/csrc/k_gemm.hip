// Gathered-row GEMM for the projections and the FFN: C[m][n] = X[m][:] . W[n][:].
//
// Each projection of a (partial) prompt pass or of a single-token decode pass
// runs over the M recomputed token rows only (Alg. 1, partial forward pass).
// M is small next to the weight matrices (1 to a few hundred rows per episode),
// so the kernel is built around streaming the packed bf16 weights once:
//  * MFMA v_mfma_f32_16x16x32_bf16 with the weight block as the A operand
//    (16 output features) and 16 token rows as the B operand; every lane loads
//    16 contiguous bytes of both operands straight from their packed layouts;
//  * one workgroup owns a PAIR of 16-row weight blocks for all the tile's
//    token rows; the pair is chosen so that the epilogue's partner values
//    sit in the same lane and register: RoPE dims (i, i + d_h/2), SwiGLU
//    (gate j, up j);
//  * weight and token fragments are prefetched a chunk ahead in registers;
//  * the k range is split across the waves of one workgroup and summed in
//    LDS in a fixed order, so results are bitwise reproducible and no
//    workgroup ever waits on another.
#include "gvc_kernels.h"
#include "gvc_sync.h"

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
  } else if (a.map == MAP_SINGLE) {
    mat_a = mat_b = 0; blk_a = blk_b = pair; b_ok = false;
  } else if (a.map == MAP_QKV_SINGLE) {
    mat_a = mat_b = pair / a.wblk[0]; blk_a = blk_b = pair % a.wblk[0]; b_ok = false;
  } else {
    mat_a = mat_b = 0;
    blk_a = 2 * pair;
    blk_b = 2 * pair + 1;
    if (blk_b >= a.wblk[0]) { blk_b = blk_a; b_ok = false; }
  }
}

__device__ __forceinline__ bf16x8 wload(const bf16x8* p) { return *p; }

__device__ __forceinline__ float silu_f(float g) { return g / (1.0f + __expf(-g)); }

// GELU, tanh form: x/2 (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3))).
__device__ __forceinline__ float gelu_f(float x) {
  return 0.5f * x * (1.0f + tanhf(0.7978845608028654f * (x + 0.044715f * x * x * x)));
}

__device__ __forceinline__ void add_bias(floatx4& v, const float* bias, int f) {
  const float4 b = *(const float4*)(bias + f);
  v[0] += b.x; v[1] += b.y; v[2] += b.z; v[3] += b.w;
}

// Epilogue of one lane: 4 consecutive output features of block A and of
// block B for token row m.  Every lane of the wave calls it (some epilogues
// shuffle across lanes); `valid` says whether row m exists (m is already
// clamped into range for address arithmetic).  rs scales the accumulators
// (folded RMSNorm, 1 otherwise).
template <int EPI>
__device__ __forceinline__ void epilogue(const GemmArgs& a, int pair, int lane, int m, floatx4 va, floatx4 vb,
                                         bool b_ok, bool valid, float rs) {
  const EpiArgs& e = a.e;
  int mat_a, blk_a, mat_b, blk_b; bool bo;
  map_pair(a, pair, mat_a, blk_a, mat_b, blk_b, bo);
  va *= rs;
  vb *= rs;
  const int sub = (lane >> 4) * 4;   // first of the 4 features this lane holds
  if constexpr (EPI == EPI_QKV) {
    if (!valid) return;
    const int dh = e.head_dim, half = dh >> 1;
    const int head = blk_a / (dh >> 4);
    const int ia = (blk_a % (dh >> 4)) * 16 + sub;   // dim within head, < half
    const int pos = e.rows.pos[m];
    const int b = e.rows.ep[m];
    if (e.bias[mat_a]) {
      add_bias(va, e.bias[mat_a], blk_a * 16 + sub);
      add_bias(vb, e.bias[mat_a], blk_b * 16 + sub);
    }
    float ra[4], rb[4];
    if (mat_a < 2 && e.rope) {
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
  } else if constexpr (EPI == EPI_QKV_RAW) {
    // single block of q, k or v for decode rows: q and k stay fp32 and
    // un-rotated (the decode attention rotates them), v goes to the cache
    if (!valid) return;
    const int f = blk_a * 16 + sub;
    if (mat_a == 0) {
      *(float4*)(e.qraw + (size_t)m * e.d + f) = float4{va[0], va[1], va[2], va[3]};
    } else if (mat_a == 1) {
      *(float4*)(e.kraw + (size_t)m * e.d + f) = float4{va[0], va[1], va[2], va[3]};
    } else {
      const int dh = e.head_dim, head = f / dh, dim = f % dh;
      bf16* v = e.vc + ((size_t)(e.rows.ep[m] * e.n_heads + head) * dh + dim) * e.kv_pad + e.rows.pos[m];
#pragma unroll
      for (int i = 0; i < 4; ++i) v[(size_t)i * e.kv_pad] = f2bf(va[i]);
    }
  } else if constexpr (EPI == EPI_RESID) {
    const int d = e.d;
    const size_t ri = (size_t)(e.resid_mapped ? e.rows.idx[m] : m) * d;
    const size_t oi = (size_t)(e.out_mapped ? e.rows.idx[m] : m) * d;
    const int fa = blk_a * 16 + sub, fb = blk_b * 16 + sub;
    if (e.bias[0]) {
      add_bias(va, e.bias[0], fa);
      if (b_ok) add_bias(vb, e.bias[0], fb);
    }
    const float4 r0 = *(const float4*)(e.resid + ri + fa);
    const float4 oa = {r0.x + va[0], r0.y + va[1], r0.z + va[2], r0.w + va[3]};
    float4 ob = {0.f, 0.f, 0.f, 0.f};
    if (b_ok) {
      const float4 r1 = *(const float4*)(e.resid + ri + fb);
      ob = float4{r1.x + vb[0], r1.y + vb[1], r1.z + vb[2], r1.w + vb[3]};
    }
    if (valid) {
      *(float4*)(e.out + oi + fa) = oa;
      if (b_ok) *(float4*)(e.out + oi + fb) = ob;
    }
    if (e.xn) {   // folded RMSNorm input of the next projection
      const float4 ga = *(const float4*)(e.xn_gain + fa);
      float ss = oa.x * oa.x + oa.y * oa.y + oa.z * oa.z + oa.w * oa.w;
      if (valid)
        *(u16x4*)(e.xn + frag_off(m, fa, e.xn_kb)) =
            u16x4{f2bf(oa.x * ga.x), f2bf(oa.y * ga.y), f2bf(oa.z * ga.z), f2bf(oa.w * ga.w)};
      if (b_ok) {
        const float4 gb = *(const float4*)(e.xn_gain + fb);
        ss += ob.x * ob.x + ob.y * ob.y + ob.z * ob.z + ob.w * ob.w;
        if (valid)
          *(u16x4*)(e.xn + frag_off(m, fb, e.xn_kb)) =
              u16x4{f2bf(ob.x * gb.x), f2bf(ob.y * gb.y), f2bf(ob.z * gb.z), f2bf(ob.w * gb.w)};
      }
      ss += __shfl_xor(ss, 16);
      ss += __shfl_xor(ss, 32);
      if (valid && lane < 16) e.ssq_out[(size_t)m * e.ssq_out_parts + pair] = ss;
    }
  } else if constexpr (EPI == EPI_SILU) {
    const int f = blk_a * 16 + sub;
    if (valid && f < e.n_feat) {
      u16x4 o;
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = f2bf(silu_f(va[i]) * vb[i]);
      *(u16x4*)(e.act + frag_off(m, f, e.kb_act)) = o;
    }
  } else if constexpr (EPI == EPI_GELU) {
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      if (half == 1 && !b_ok) break;
      const int f = (half ? blk_b : blk_a) * 16 + sub;
      floatx4 v = half ? vb : va;
      if (!valid || f >= e.n_feat) continue;
      if (e.bias[0]) add_bias(v, e.bias[0], f);
      const u16x4 o = {f2bf(gelu_f(v[0])), f2bf(gelu_f(v[1])), f2bf(gelu_f(v[2])), f2bf(gelu_f(v[3]))};
      *(u16x4*)(e.act + frag_off(m, f, e.kb_act)) = o;
    }
  } else if constexpr (EPI == EPI_PATCH) {
    if (!valid) return;
    const float inv255 = 1.0f / 255.0f;
    float* o = e.store + (size_t)m * e.ld_store;
    const float* pt = e.pos_tab + (size_t)e.rows.pos[m] * e.ld_store;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      if (half == 1 && !b_ok) break;
      const int f = (half ? blk_b : blk_a) * 16 + sub;
      const floatx4& v = half ? vb : va;
      const float4 bb = *(const float4*)(e.bias[0] + f), pp = *(const float4*)(pt + f);
      *(float4*)(o + f) = float4{v[0] * inv255 + bb.x + pp.x, v[1] * inv255 + bb.y + pp.y,
                                 v[2] * inv255 + bb.z + pp.z, v[3] * inv255 + bb.w + pp.w};
    }
  } else if constexpr (EPI == EPI_STORE) {
    if (!valid) return;
    float* o = e.store + (size_t)m * e.ld_store;
    const int fa = blk_a * 16 + sub;
    if (fa < a.n_out) *(float4*)(o + fa) = float4{va[0], va[1], va[2], va[3]};
    const int fb = blk_b * 16 + sub;
    if (b_ok && fb < a.n_out) *(float4*)(o + fb) = float4{vb[0], vb[1], vb[2], vb[3]};
  } else {  // EPI_EMBED
    if (!valid) return;
    const int d = e.d;
    const int pos = e.rows.pos[m], b = e.rows.ep[m];
    float* h = e.h0 + (size_t)e.rows.idx[m] * d;
    const float sc = e.vis_scale;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      if (half == 1 && !b_ok) break;
      const int f = (half ? blk_b : blk_a) * 16 + sub;
      const floatx4& v = half ? vb : va;
      float4 o;
      if (pos >= 1 && pos <= e.n_patches) {
        o.x = v[0] * sc; o.y = v[1] * sc; o.z = v[2] * sc; o.w = v[3] * sc;
        if (e.bias[0]) {
          const float4 bb = *(const float4*)(e.bias[0] + f);
          o.x += bb.x; o.y += bb.y; o.z += bb.z; o.w += bb.w;
        }
      } else if (pos < e.n_patches + e.n_text) {
        const int t = pos == 0 ? 0 : pos - e.n_patches;
        const bf16* er = e.embed + (size_t)min(max(e.text_ids[b * e.n_text + t], 0), e.n_vocab - 1) * d + f;
        o.x = bf2f(er[0]); o.y = bf2f(er[1]); o.z = bf2f(er[2]); o.w = bf2f(er[3]);
      } else {
        const float* xr = e.extra + ((size_t)b * e.n_extra + (pos - e.n_patches - e.n_text)) * d + f;
        o = *(const float4*)xr;
      }
      *(float4*)(h + f) = o;
    }
  }
}

// One workgroup owns one pair of weight blocks (one block for the single
// maps) and a tile of KT x NT blocks of 16 token rows.  Its KT * KS waves are
// KT token groups (NT blocks each) times KS shares of the k range: the waves
// of one k share read the same weight fragments at the same time, so the
// weights leave HBM once per workgroup while each wave keeps only NT token
// blocks in registers.  The k shares are summed through LDS in a fixed order
// (deterministic, no cross-workgroup traffic).  Each wave streams its share
// in chunks of PF k-steps, double-buffered in registers with no branch
// between a chunk's loads and its MFMAs, so two chunks are in flight; the
// prefetch of the chunk after the last re-reads the last chunk instead of
// branching.  Token fragments come straight from the (L2-resident)
// activations.
template <int KS, int KT, int NT, int PF, int EPI, bool ONE>
__global__ __launch_bounds__(KS * KT * 64) void k_gemm_ks(const GemmArgs a) {
  constexpr int KW = KS * KT;
  __shared__ floatx4 red[KW][2][64];
  __shared__ float ssq_red[KW][16];
  __shared__ float rscale[16];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tg = wave / KS, ks = wave % KS;
  // XCD-aware order: workgroup ids go round-robin over the 8 XCDs, so the
  // token tiles of one work unit get ids 8 apart -- same XCD, dispatched
  // together -- and the later tiles find the unit's weights in that L2.
  const int grp = blockIdx.x / (8 * a.mtiles), r8 = blockIdx.x % (8 * a.mtiles);
  const int pair = grp * 8 + (r8 & 7), mt = r8 >> 3;
  if (pair >= a.n_pairs) return;
  // Folded RMSNorm (single token block): lane (row r = lane % 16, chunk
  // wave * 4 + lane / 16) loads up to SQ of the row's partial sums of squares
  // now and adds them after the main loop, so the loads overlap the stream.
  constexpr int SQ = 16;
  float sq[SQ];
  const bool fold = NT == 1 && KT == 1 && a.e.ssq_in != nullptr;
  if (fold) {
    const int r = min(lane & 15, a.M - 1);
    const int nch = KW * 4, ch = wave * 4 + (lane >> 4);
    const int per = (a.e.ssq_parts + nch - 1) / nch;
    const float* sp = a.e.ssq_in + (size_t)r * a.e.ssq_parts;
#pragma unroll
    for (int i = 0; i < SQ; ++i) {
      const int idx = ch * per + i;
      const float v = sp[min(idx, a.e.ssq_parts - 1)];
      sq[i] = (i < per && idx < a.e.ssq_parts) ? v : 0.f;
    }
  }
  int mat_a, blk_a, mat_b, blk_b; bool b_ok;
  map_pair(a, pair, mat_a, blk_a, mat_b, blk_b, b_ok);
  const bf16x8* wa = a.w[mat_a] + (size_t)blk_a * a.KB * 64 + lane;
  const bf16x8* wb = a.w[mat_b] + (size_t)blk_b * a.KB * 64 + lane;
  const int mb0 = (mt * KT + tg) * NT;   // first token block of this wave
  // Lanes of token rows >= M re-read the last valid row of their block:
  // those output columns are never stored, and the shared address keeps a
  // decode launch (M = 1) from fetching 15 padding rows per fragment.
  const bf16x8* xg[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int mb = min(mb0 + t, a.mblocks - 1);
    const int xl = (lane & 48) | min(lane & 15, a.M - 1 - mb * 16);
    xg[t] = a.x + (size_t)mb * a.KB * 64 + xl;
  }
  // this wave's contiguous share of the k range
  const int kb0 = min(a.KB, ks * a.kb_per_split);
  const int nsteps = min(a.KB, kb0 + a.kb_per_split) - kb0;
  const int nchunks = nsteps / PF;

  floatx4 acc_a[NT], acc_b[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) { acc_a[t] = floatx4{0, 0, 0, 0}; acc_b[t] = floatx4{0, 0, 0, 0}; }
  bf16x8 a0[PF], b0[PF], x0[PF][NT], a1[PF], b1[PF], x1[PF][NT];
  auto load = [&](bf16x8 (&A)[PF], bf16x8 (&Bv)[PF], bf16x8 (&X)[PF][NT], int c) {
    const size_t kb = (size_t)(kb0 + min(c, nchunks - 1) * PF) * 64;
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      const size_t o = kb + (size_t)p * 64;
      A[p] = wa[o];
      if constexpr (!ONE) Bv[p] = wb[o];
#pragma unroll
      for (int t = 0; t < NT; ++t) X[p][t] = xg[t][o];
    }
  };
  auto compute = [&](const bf16x8 (&A)[PF], const bf16x8 (&Bv)[PF], const bf16x8 (&X)[PF][NT]) {
#pragma unroll
    for (int p = 0; p < PF; ++p)
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        acc_a[t] = mfma16(A[p], X[p][t], acc_a[t]);
        if constexpr (!ONE) acc_b[t] = mfma16(Bv[p], X[p][t], acc_b[t]);
      }
  };
  if (nchunks > 0) {
    load(a0, b0, x0, 0);
    int c = 0;
    for (; c + 1 < nchunks; c += 2) {
      load(a1, b1, x1, c + 1);
      compute(a0, b0, x0);
      load(a0, b0, x0, c + 2);
      compute(a1, b1, x1);
    }
    if (c < nchunks) compute(a0, b0, x0);
  }
  for (int s = nchunks * PF; s < nsteps; ++s) {   // ragged k tail
    const size_t kb = (size_t)(kb0 + s) * 64;
    const bf16x8 wva = wa[kb];
    const bf16x8 wvb = ONE ? wva : wb[kb];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const bf16x8 xv = xg[t][kb];
      acc_a[t] = mfma16(wva, xv, acc_a[t]);
      if constexpr (!ONE) acc_b[t] = mfma16(wvb, xv, acc_b[t]);
    }
  }
  if (fold) {
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < SQ; ++i) t += sq[i];
    t += __shfl_xor(t, 16);
    t += __shfl_xor(t, 32);
    if (lane < 16) ssq_red[wave][lane] = t;
    __syncthreads();
    if (wave == 0 && lane < 16) {
      float u = ssq_red[0][lane];
#pragma unroll
      for (int w = 1; w < KW; ++w) u += ssq_red[w][lane];
      rscale[lane] = 1.0f / sqrtf(u / (float)a.e.norm_dim + a.e.norm_eps);
    }
  }
  // Reduce over the KS k shares of each token group, one token block per
  // round; the wave with ks == t % KS keeps the sum of block t and runs its
  // epilogue.
  const int col = lane & 15;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    red[wave][0][lane] = acc_a[t];
    if constexpr (!ONE) red[wave][1][lane] = acc_b[t];
    __syncthreads();
    if (ks == t % KS) {
      floatx4 sa = red[tg * KS][0][lane], sb = ONE ? sa : red[tg * KS][1][lane];
#pragma unroll
      for (int w = 1; w < KS; ++w) {
        sa += red[tg * KS + w][0][lane];
        if constexpr (!ONE) sb += red[tg * KS + w][1][lane];
      }
      acc_a[t] = sa; acc_b[t] = sb;
    }
    __syncthreads();
  }
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    if (ks != t % KS) continue;
    const int m = (mb0 + t) * 16 + col;
    const float rs = fold ? rscale[col] : 1.0f;
    epilogue<EPI>(a, pair, lane, min(m, a.M - 1), acc_a[t], acc_b[t], b_ok, m < a.M, rs);
  }
}

// Many-row variant (batched episodes: thousands of rows, MFMA-bound).  A
// workgroup of 8 waves owns kBigPairs weight pairs x 4 TW blocks of 16
// token rows and walks the whole k range; every k step, both operands'
// fragments for the tile (2 kBigPairs weight + 4 TW token fragments) are
// copied straight into LDS (global_load_lds), three stages deep so one step
// is in flight while another is read, with one workgroup barrier per step.
// Wave (wp, wt) multiplies pairs wp*2..wp*2+1 by token blocks
// wt*TW..wt*TW+TW-1 (4 TW MFMAs per k step from 4 + TW LDS fragment reads)
// and runs the same fused epilogue as k_gemm_ks.  Each row's sum runs over
// k in order, so a row's result does not depend on the tile it falls in or
// on the tile height (TW = 4, 3, 2: 256-, 192-, 128-row tiles; the launcher
// picks one per launch).
constexpr int kBigWP = 2, kBigWT = 4, kBigPW = 2;
constexpr int kBigPairs = kBigWP * kBigPW;
constexpr int kBigStages = 3;
template <int TW>
constexpr int big_frags() { return 2 * kBigPairs + kBigWT * TW; }   // fragments per k step
template <int TW>
constexpr int big_lds_bytes() { return kBigStages * big_frags<TW>() * 1024; }

typedef unsigned u32x4b __attribute__((ext_vector_type(4)));
#define GPB(p) ((const void __attribute__((address_space(1)))*)(p))
#define LPB(p) ((void __attribute__((address_space(3)))*)(p))

template <int N>
__device__ __forceinline__ void big_wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

template <int EPI, int TW>
__global__ __launch_bounds__(kBigWP * kBigWT * 64) void k_gemm_big(const GemmArgs a) {
  constexpr int NW = kBigWP * kBigWT;
  constexpr int WF = 2 * kBigPairs;
  constexpr int FR = big_frags<TW>();
  constexpr int LPW = (FR + NW - 1) / NW;          // fragment copies per wave per k step
  extern __shared__ u32x4b big_lds[];              // [kBigStages][FR][64]
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wp = wv % kBigWP, wt = wv / kBigWP;
  // XCD-aware order: all tiles of one weight tile run on XCD (tile % 8) and
  // share its weights in that L2; within an XCD, jobs run in groups of 8
  // token tiles x all of the XCD's weight tiles, so the workgroups resident
  // at one time share both operands' tiles
  const int x = blockIdx.x, xcd = x & 7, i = x >> 3;
  const int ntiles = (a.n_pairs + kBigPairs - 1) / kBigPairs;
  const int nnt = (ntiles + 7) / 8, g = i / (8 * nnt), r = i % (8 * nnt);
  const int gs = min(8, a.mtiles - g * 8);
  const int nt = xcd + 8 * (r / gs), mt = g * 8 + r % gs;
  if (nt >= ntiles) return;
  const int pair0 = nt * kBigPairs, tb0 = mt * kBigWT * TW;
  const bf16x8* src[LPW];
  int dst[LPW];
#pragma unroll
  for (int l = 0; l < LPW; ++l) {
    const int f = min(wv + l * NW, FR - 1);
    dst[l] = f;
    if (f < WF) {
      int ma, ba, mb, bb; bool ok;
      map_pair(a, min(pair0 + f / 2, a.n_pairs - 1), ma, ba, mb, bb, ok);
      src[l] = (f & 1) ? a.w[mb] + (size_t)bb * a.KB * 64 + lane : a.w[ma] + (size_t)ba * a.KB * 64 + lane;
    } else {
      src[l] = a.x + (size_t)min(tb0 + f - WF, a.mblocks - 1) * a.KB * 64 + lane;
    }
  }
  auto issue = [&](int k) {   // k steps past the end re-read the last one (in bounds)
    u32x4b* st = big_lds + (k % kBigStages) * FR * 64;
    const size_t o = (size_t)min(k, a.KB - 1) * 64;
#pragma unroll
    for (int l = 0; l < LPW; ++l) __builtin_amdgcn_global_load_lds(GPB(src[l] + o), LPB(st + dst[l] * 64), 16, 0, 0);
  };
  floatx4 acc[2 * kBigPW][TW];
#pragma unroll
  for (int p = 0; p < 2 * kBigPW; ++p)
#pragma unroll
    for (int j = 0; j < TW; ++j) acc[p][j] = floatx4{0, 0, 0, 0};
  issue(0);
  for (int k = 0; k < a.KB; ++k) {
    // stage (k + 1) % 3 last held step k - 2, which every wave finished
    // before the barrier of step k - 1
    issue(k + 1);
    big_wait_vm<LPW>();
    lds_barrier();
    const u32x4b* st = big_lds + (k % kBigStages) * FR * 64;
    bf16x8 wf[2 * kBigPW], xf[TW];
#pragma unroll
    for (int p = 0; p < 2 * kBigPW; ++p) wf[p] = __builtin_bit_cast(bf16x8, st[(2 * wp * kBigPW + p) * 64 + lane]);
#pragma unroll
    for (int j = 0; j < TW; ++j) xf[j] = __builtin_bit_cast(bf16x8, st[(WF + wt * TW + j) * 64 + lane]);
#pragma unroll
    for (int j = 0; j < TW; ++j)
#pragma unroll
      for (int p = 0; p < 2 * kBigPW; ++p) acc[p][j] = mfma16(wf[p], xf[j], acc[p][j]);
  }
  big_wait_vm<0>();
  const int col = lane & 15;
#pragma unroll
  for (int p = 0; p < kBigPW; ++p) {
    const int pair = pair0 + wp * kBigPW + p;
    if (pair >= a.n_pairs) continue;
    int ma, ba, mb, bb; bool b_ok;
    map_pair(a, pair, ma, ba, mb, bb, b_ok);
#pragma unroll
    for (int j = 0; j < TW; ++j) {
      const int m = (tb0 + wt * TW + j) * 16 + col;
      epilogue<EPI>(a, pair, lane, min(m, a.M - 1), acc[2 * p][j], acc[2 * p + 1][j], b_ok, m < a.M, 1.0f);
    }
  }
}

template <int EPI, int TW>
static hipError_t launch_big_tw(GemmArgs a, hipStream_t s) {
  static bool attr = false;
  if (!attr) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemm_big<EPI, TW>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, big_lds_bytes<TW>());
    if (e != hipSuccess) return e;
    attr = true;
  }
  a.mtiles = (a.mblocks + kBigWT * TW - 1) / (kBigWT * TW);
  const int ntiles = (a.n_pairs + kBigPairs - 1) / kBigPairs;
  const dim3 grid(8 * ((ntiles + 7) / 8) * a.mtiles);
  hipLaunchKernelGGL((k_gemm_big<EPI, TW>), grid, dim3(kBigWP * kBigWT * 64), big_lds_bytes<TW>(), s, a);
  return hipGetLastError();
}

// Tile height: a launch takes about ceil(workgroups / resident) rounds of
// one workgroup's k loop.  Two 256-row workgroups fit a CU (72 KiB of LDS
// each), two 192-row ones (60 KiB), three 128-row ones (48 KiB); on the 7B
// projections at 736-4416 rows a round of 128-row tiles measured 0.885 of a
// 256-row round and, on the output, down and QKV projections, a round of
// 192-row tiles 0.87.  192-row tiles are only taken for launches of at most
// 96 weight tiles that would give more than one 128-row workgroup per CU
// (gate/up and smaller launches measured faster on the other two).
template <int EPI>
static hipError_t launch_big_epi(const GemmArgs& a, hipStream_t s) {
  static int cus = 0;
  if (!cus) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    if (cus <= 0) return hipErrorInvalidDevice;
  }
  const long long ntiles = (a.n_pairs + kBigPairs - 1) / kBigPairs;
  const long long j4 = ntiles * ((a.mblocks + 4 * kBigWT - 1) / (4 * kBigWT));
  const long long j2 = ntiles * ((a.mblocks + 2 * kBigWT - 1) / (2 * kBigWT));
  const long long j3 = ntiles * ((a.mblocks + 3 * kBigWT - 1) / (3 * kBigWT));
  const long long r4 = (j4 + 2LL * cus - 1) / (2LL * cus), r2 = (j2 + 3LL * cus - 1) / (3LL * cus);
  const long long r3 = (j3 + 2LL * cus - 1) / (2LL * cus);
  long long best = 1000 * r4;
  int tw = 4;
  if (885 * r2 < best) { best = 885 * r2; tw = 2; }
  if (ntiles <= 96 && j2 > cus && 870 * r3 < best) tw = 3;
  if (a.big_tw >= 2 && a.big_tw <= 4) tw = a.big_tw;   // fixed by the caller (testing)
  if (tw == 3) return launch_big_tw<EPI, 3>(a, s);
  if (tw == 2) return launch_big_tw<EPI, 2>(a, s);
  return launch_big_tw<EPI, 4>(a, s);
}

// Tiles are chosen here from a.mblocks; pair maps only, no folded norm.
hipError_t launch_gemm_big(const GemmArgs& a, int epi, hipStream_t s) {
  if (a.map == MAP_SINGLE || a.map == MAP_QKV_SINGLE || a.e.ssq_in) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_QKV: return launch_big_epi<EPI_QKV>(a, s);
    case EPI_RESID: return launch_big_epi<EPI_RESID>(a, s);
    case EPI_SILU: return launch_big_epi<EPI_SILU>(a, s);
    case EPI_STORE: return launch_big_epi<EPI_STORE>(a, s);
    case EPI_EMBED: return launch_big_epi<EPI_EMBED>(a, s);
    case EPI_PATCH: return launch_big_epi<EPI_PATCH>(a, s);
    case EPI_GELU: return launch_big_epi<EPI_GELU>(a, s);
    default: return hipErrorInvalidValue;
  }
}

// Split-k variant for a large prompt-pass projection at a few hundred rows
// (the 7B gate/up projection at batch 1).  The per-pair
// kernel reads each token fragment once per weight pair, so its L2 -> CU
// traffic is several times the weight bytes; here a workgroup of 8 waves
// owns 8 * NBW consecutive weight blocks (of all the launch's matrices, in
// order) for one k slice and one tile of T token blocks, and the tile's
// token fragments pass through LDS once for all 8 waves.  Per chunk of KC k
// steps the waves copy the token fragments straight into LDS
// (global_load_lds) D chunks ahead, D + 2 stages deep (the stage written at
// chunk c last held chunk c - 2, which every wave finished before the
// barrier of chunk c - 1), and each wave loads its NBW weight fragments into
// registers D chunks ahead.  Partial sums go to part[slice][row][feature];
// k_gemm_sk_epi then adds the slices in order and runs the fused epilogue.
// The slices depend only on the matrix shape, so a row's result never
// depends on how many rows a pass recomputes.
template <int T, int NBW, int KC, int D>
__global__ __launch_bounds__(8 * 64) void k_gemm_sk(const GemmArgs a) {
  constexpr int NW = 8;
  constexpr int NF = KC * T;                       // token fragments per chunk
  constexpr int ITOK = (NF + NW - 1) / NW;         // copies per wave per chunk (duplicates pad the last)
  constexpr int IW = KC * NBW;
  constexpr int NST = D + 2;
  static_assert(D * (ITOK + IW) < 64, "vmcnt range");
  extern __shared__ u32x4b sk_lds[];               // [NST][KC][T][64]
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int id = blockIdx.x;
  const int g = id % a.sk_groups;
  id /= a.sk_groups;
  const int s = id % a.sk_slices, mt = id / a.sk_slices;
  const int kb0 = s * a.sk_steps, nk = min(a.KB, kb0 + a.sk_steps) - kb0;
  if (nk <= 0) return;
  const int mb0 = mt * T, nT = min(T, a.mblocks - mb0);
  const int nblk = a.wblk[0] * (a.map == MAP_QKV ? 3 : (a.map == MAP_GU ? 2 : 1));
  const bf16x8* wp[NBW];
  int vbs[NBW];
#pragma unroll
  for (int j = 0; j < NBW; ++j) {
    const int vb = (g * NW + wv) * NBW + j;
    vbs[j] = vb;
    const int vc = min(vb, nblk - 1), mat = vc / a.wblk[0], blk = vc % a.wblk[0];
    wp[j] = a.w[mat] + ((size_t)blk * a.KB + kb0) * 64 + lane;
  }
  const int nchunks = (nk + KC - 1) / KC;
  auto issue_tok = [&](int c) {   // chunks past the end re-read the last k step (in bounds)
    u32x4b* buf = sk_lds + (c % NST) * NF * 64;
#pragma unroll
    for (int i = 0; i < ITOK; ++i) {
      const int f = min(wv + i * NW, NF - 1), kk = f / T, t = f % T;
      const int kb = kb0 + min(c * KC + kk, nk - 1);
      const int tb = mb0 + min(t, nT - 1);
      __builtin_amdgcn_global_load_lds(GPB(a.x + ((size_t)tb * a.KB + kb) * 64 + lane), LPB(buf + f * 64), 16, 0, 0);
    }
  };
  bf16x8 wb[D + 1][KC][NBW];
  auto issue_w = [&](int c, bf16x8 (&W)[KC][NBW]) {
#pragma unroll
    for (int kk = 0; kk < KC; ++kk) {
      const size_t k = (size_t)min(c * KC + kk, nk - 1) * 64;
#pragma unroll
      for (int j = 0; j < NBW; ++j) W[kk][j] = wp[j][k];
    }
  };
  floatx4 acc[NBW][T];
#pragma unroll
  for (int j = 0; j < NBW; ++j)
#pragma unroll
    for (int t = 0; t < T; ++t) acc[j][t] = floatx4{0, 0, 0, 0};
#pragma unroll
  for (int u = 0; u < D; ++u) {
    issue_tok(u);
    issue_w(u, wb[u]);
  }
  for (int c0 = 0; c0 < nchunks; c0 += D + 1) {
#pragma unroll
    for (int u = 0; u <= D; ++u) {
      const int c = c0 + u;
      if (c < nchunks) {
        issue_tok(c + D);
        issue_w(c + D, wb[(u + D) % (D + 1)]);
        big_wait_vm<D * (ITOK + IW)>();
        lds_barrier();
        const u32x4b* buf = sk_lds + (c % NST) * NF * 64;
#pragma unroll
        for (int kk = 0; kk < KC; ++kk) {
          if (c * KC + kk < nk) {
#pragma unroll
            for (int t = 0; t < T; ++t) {
              const bf16x8 xf = __builtin_bit_cast(bf16x8, buf[(kk * T + t) * 64 + lane]);
#pragma unroll
              for (int j = 0; j < NBW; ++j) acc[j][t] = mfma16(wb[u][kk][j], xf, acc[j][t]);
            }
          }
        }
      }
    }
  }
  big_wait_vm<0>();
  const int col = lane & 15, sub = (lane >> 4) * 4;
#pragma unroll
  for (int j = 0; j < NBW; ++j) {
    if (vbs[j] >= nblk) continue;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      if (t >= nT) continue;
      const int m = (mb0 + t) * 16 + col;
      if (m < a.M) *(floatx4*)(a.part + ((size_t)s * a.part_rows + m) * a.part_ld + vbs[j] * 16 + sub) = acc[j][t];
    }
  }
}

// Split-k core with decoupled operand streams (the partial layout of
// k_gemm_sk; with NCW = 8, PB = 2 also its work split): NCW compute waves each
// stream their PB weight blocks through a private LDS ring of RW fragments (non-temporal
// direct-to-LDS loads, in k order), and NXW loader waves copy the tile's
// token fragments into DX LDS stages of KC k steps.  Weight loads then never
// queue behind token loads in a wave's in-order memory counter, and a
// compute wave waits only for its own oldest weight fragment; one workgroup
// barrier per chunk hands the token stages over (the stage refilled after
// the barrier of chunk c last held chunk c - 1, which every compute wave
// finished before arriving).
template <int T, int NCW, int PB, int KC, int DX, int NXW, int RW>
__global__ __launch_bounds__((NCW + NXW) * 64) void k_gemm_dx(const GemmArgs a) {
  constexpr int NF = KC * T, ITOK = (NF + NXW - 1) / NXW;
  static_assert((DX - 2) * ITOK < 64 && RW < 64, "vmcnt range");
  extern __shared__ u32x4b dx_lds[];                 // [NCW][RW][64] rings, then [DX][NF][64] token stages
  u32x4b* const xst = dx_lds + NCW * RW * 64;
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int id = blockIdx.x;
  const int g = id % a.sk_groups;
  id /= a.sk_groups;
  const int s = id % a.sk_slices, mt = id / a.sk_slices;
  const int kb0 = s * a.sk_steps, nk = min(a.KB, kb0 + a.sk_steps) - kb0;
  if (nk <= 0) return;
  const int nch = (nk + KC - 1) / KC;
  const int mb0 = mt * T, nT = min(T, a.mblocks - mb0);
  const int nblk = a.wblk[0] * (a.map == MAP_QKV ? 3 : (a.map == MAP_GU ? 2 : 1));
  if (wv >= NCW) {   // token loader
    const int x = wv - NCW;
    auto issue = [&](int c) {   // chunks past the end re-read the last k step (in bounds)
      u32x4b* st = xst + (c % DX) * NF * 64;
#pragma unroll
      for (int i = 0; i < ITOK; ++i) {
        const int f = min(x + i * NXW, NF - 1), kk = f / T, t = f % T;
        const int kb = kb0 + min(c * KC + kk, nk - 1);
        __builtin_amdgcn_global_load_lds(GPB(a.x + ((size_t)(mb0 + min(t, nT - 1)) * a.KB + kb) * 64 + lane),
                                         LPB(st + f * 64), 16, 0, 0);
      }
    };
#pragma unroll
    for (int c = 0; c < DX - 1; ++c) issue(c);
    for (int c = 0; c < nch; ++c) {
      big_wait_vm<(DX - 2) * ITOK>();
      lds_barrier();
      issue(c + DX - 1);
    }
    big_wait_vm<0>();
    return;
  }
  const bf16x8* wp[PB];
  int vbs[PB];
#pragma unroll
  for (int p = 0; p < PB; ++p) {
    const int vb = (g * NCW + wv) * PB + p;
    vbs[p] = vb;
    const int vc = min(vb, nblk - 1), mat = vc / a.wblk[0], blk = vc % a.wblk[0];
    wp[p] = a.w[mat] + ((size_t)blk * a.KB + kb0) * 64 + lane;
  }
  u32x4b* const ring = dx_lds + wv * RW * 64;
  const int total = nk * PB;
  int next = 0;   // next fragment of this wave's stream (k major, block minor)
  auto refill = [&](int slot) {
    const int i = min(next, total - 1), k = i / PB, p = i - k * PB;
    const bf16x8* src = wp[0];
#pragma unroll
    for (int q = 1; q < PB; ++q)
      if (p == q) src = wp[q];
    __builtin_amdgcn_global_load_lds(GPB(src + (size_t)k * 64), LPB(ring + slot * 64), 16, 0, 2);
    ++next;
  };
#pragma unroll
  for (int r = 0; r < RW; ++r) refill(r);
  floatx4 acc[PB][T];
#pragma unroll
  for (int p = 0; p < PB; ++p)
#pragma unroll
    for (int t = 0; t < T; ++t) acc[p][t] = floatx4{0, 0, 0, 0};
  int slot = 0;
  for (int c = 0; c < nch; ++c) {
    lds_barrier();
    const u32x4b* st = xst + (c % DX) * NF * 64;
#pragma unroll
    for (int kk = 0; kk < KC; ++kk) {
      if (c * KC + kk >= nk) break;
      bf16x8 wf[PB];
#pragma unroll
      for (int p = 0; p < PB; ++p) {
        big_wait_vm<RW - 1>();
        wf[p] = __builtin_bit_cast(bf16x8, ring[slot * 64 + lane]);
        __builtin_amdgcn_s_waitcnt(0xC07F);   // the read has left the slot before it is refilled
        refill(slot);
        slot = slot + 1 == RW ? 0 : slot + 1;
      }
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const bf16x8 xf = __builtin_bit_cast(bf16x8, st[(kk * T + t) * 64 + lane]);
#pragma unroll
        for (int p = 0; p < PB; ++p) acc[p][t] = mfma16(wf[p], xf, acc[p][t]);
      }
    }
  }
  big_wait_vm<0>();
  const int col = lane & 15, sub = (lane >> 4) * 4;
#pragma unroll
  for (int p = 0; p < PB; ++p) {
    if (vbs[p] >= nblk) continue;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      if (t >= nT) continue;
      const int m = (mb0 + t) * 16 + col;
      if (m < a.M)   // rows past the last one are never summed
        *(floatx4*)(a.part + ((size_t)s * a.part_rows + m) * a.part_ld + vbs[p] * 16 + sub) = acc[p][t];
    }
  }
}

// Sums the k slices of k_gemm_sk in order and runs the epilogue: one wave
// per (work pair, block of 16 rows), in the lane layout of the MFMA result.
// The 4 waves of a workgroup take 4 consecutive pairs of one row block, so
// each row's partial sums are read as whole cache lines by one CU (C2
// gate/up: prompt pass 6.56 -> 6.48 ms against row-block-minor order).
template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_sk_epi(const GemmArgs a) {
  const int lane = threadIdx.x & 63;
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (w >= a.n_pairs * a.mblocks) return;
  const int pair = w % a.n_pairs, mb = w / a.n_pairs;
  int ma, ba, mb2, bb; bool b_ok;
  map_pair(a, pair, ma, ba, mb2, bb, b_ok);
  const int m = mb * 16 + (lane & 15), sub = (lane >> 4) * 4;
  const int fa = (ma * a.wblk[0] + ba) * 16 + sub, fb = (mb2 * a.wblk[0] + bb) * 16 + sub;
  floatx4 va = {0, 0, 0, 0}, vb = {0, 0, 0, 0};
  if (m < a.M)   // the cores store no partial sums for rows past the last one
    for (int s = 0; s < a.sk_slices; ++s) {
      const float* row = a.part + ((size_t)s * a.part_rows + m) * a.part_ld;
      va += *(const floatx4*)(row + fa);
      if (b_ok) vb += *(const floatx4*)(row + fb);
    }
  epilogue<EPI>(a, pair, lane, min(m, a.M - 1), va, vb, b_ok, m < a.M, 1.0f);
}

template <int T, int NBW, int KC, int D>
static hipError_t launch_sk_core(const GemmArgs& a, hipStream_t s) {
  constexpr int lds = (D + 2) * KC * T * 1024;
  static bool attr = false;
  if (!attr) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemm_sk<T, NBW, KC, D>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int mtiles = (a.mblocks + T - 1) / T;
  hipLaunchKernelGGL((k_gemm_sk<T, NBW, KC, D>), dim3(a.sk_groups * a.sk_slices * mtiles), dim3(8 * 64), lds, s, a);
  return hipGetLastError();
}

template <int EPI>
static hipError_t launch_sk_epi(const GemmArgs& a, hipStream_t s) {
  const int waves = a.n_pairs * a.mblocks;
  hipLaunchKernelGGL(k_gemm_sk_epi<EPI>, dim3((waves + 3) / 4), dim3(256), 0, s, a);
  return hipGetLastError();
}

// Tiles of 10 token blocks, 2 weight blocks per wave (16 per workgroup),
// chunks of 4 k steps, one chunk ahead.
constexpr int kSkT = 10, kSkNBW = 2, kSkKC = 4, kSkD = 1;
// Decoupled core: the same 16-block groups, chunks of 2 k steps in 4 token
// stages, 2 loader waves, weight rings of 8 fragments (144 KiB of LDS).
// Measured on the 7B gate/up projection at 148 rows: prompt pass 6.58 ms
// against 6.80 with k_gemm_sk (4 or 8 loader waves, 12-fragment rings or
// 4-step chunks: within 0.05 ms).  On QKV (2 or 4 slices) and the down
// projection (8 or 16) it does not beat the per-pair kernel.
constexpr int kDxKC = 2, kDxD = 4, kDxNXW = 2, kDxRW = 8;
// Wide and narrow projections (QKV; down): one weight block per compute wave,
// so that a launch of whole k slices fills the 256 compute units with one
// workgroup each -- QKV 64 groups of 12 blocks x 4 slices, down 32 groups of
// 8 blocks x 8 slices.  The wide core has 12 compute waves and 3 token stages
// (156 KiB of LDS).
constexpr int kDxWideW = 12, kDxWideD = 4, kDxWideR = 6, kDxNarrowW = 8;
// Tall tiles: a launch of 11-18 token blocks (161-288 rows) as one tile of
// 18 blocks per k slice, so each slice's weights leave HBM once instead of
// once per 160-row tile (two rounds of workgroups, each streaming them
// again).  The taller token stages fit beside the rings with 3 stages and
// 4-fragment rings in the wide shape (156 KiB of LDS), 2 stages in the narrow
// one (136 KiB); 1-step chunks in 3-4 stages, 4 loader waves, 8-fragment
// rings and a separate 14-block tile measured within 1%.  A slice's partial
// sums are the same MFMA sequence in either tiling, so they are bit-identical.
constexpr int kSkTallT = 18, kDxTallWideD = 3, kDxTallWideR = 4, kDxTallNarrowD = 2;

template <int T, int NCW, int PB, int KC, int DX, int NXW, int RW>
static hipError_t launch_dx_core(const GemmArgs& a, hipStream_t s) {
  constexpr int lds = (NCW * RW + DX * KC * T) * 1024;
  static_assert(lds <= 160 * 1024, "LDS");
  static bool attr = false;
  if (!attr) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemm_dx<T, NCW, PB, KC, DX, NXW, RW>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int mtiles = (a.mblocks + T - 1) / T;
  hipLaunchKernelGGL((k_gemm_dx<T, NCW, PB, KC, DX, NXW, RW>), dim3(a.sk_groups * a.sk_slices * mtiles),
                     dim3((NCW + NXW) * 64), lds, s, a);
  return hipGetLastError();
}

bool gemm_sk_tall_rows(int M) {
  const int mblocks = (M + 15) / 16;
  return mblocks > kSkT && mblocks <= kSkTallT;
}

int gemm_sk_group_blocks(int sk_shape) {
  return sk_shape == SK_WIDE ? kDxWideW : (sk_shape == SK_NARROW ? kDxNarrowW : 8 * kSkNBW);
}

hipError_t launch_gemm_sk(const GemmArgs& a, int epi, hipStream_t s) {
  if (a.map == MAP_SINGLE || a.map == MAP_QKV_SINGLE || a.e.ssq_in || !a.part) return hipErrorInvalidValue;
  if (a.sk_shape != SK_GU && !a.sk_dx) return hipErrorInvalidValue;   // one-block shapes exist for k_gemm_dx only
  const bool tall = a.sk_tall && gemm_sk_tall_rows(a.M);
  hipError_t e;
  if (a.sk_shape == SK_WIDE)
    e = tall ? launch_dx_core<kSkTallT, kDxWideW, 1, kDxKC, kDxTallWideD, kDxNXW, kDxTallWideR>(a, s)
             : launch_dx_core<kSkT, kDxWideW, 1, kDxKC, kDxWideD, kDxNXW, kDxWideR>(a, s);
  else if (a.sk_shape == SK_NARROW)
    e = tall ? launch_dx_core<kSkTallT, kDxNarrowW, 1, kDxKC, kDxTallNarrowD, kDxNXW, kDxRW>(a, s)
             : launch_dx_core<kSkT, kDxNarrowW, 1, kDxKC, kDxD, kDxNXW, kDxRW>(a, s);
  else
    e = a.sk_dx ? launch_dx_core<kSkT, 8, kSkNBW, kDxKC, kDxD, kDxNXW, kDxRW>(a, s)
                : launch_sk_core<kSkT, kSkNBW, kSkKC, kSkD>(a, s);
  if (e != hipSuccess) return e;
  switch (epi) {
    case EPI_QKV: return launch_sk_epi<EPI_QKV>(a, s);
    case EPI_RESID: return launch_sk_epi<EPI_RESID>(a, s);
    case EPI_SILU: return launch_sk_epi<EPI_SILU>(a, s);
    default: return hipErrorInvalidValue;
  }
}

template <int EPI, int KT, int NT, bool ONE>
static hipError_t launch_one(const GemmArgs& a, hipStream_t s) {
  constexpr int PF = gemm_pf(NT);
  const dim3 grid((a.n_pairs + 7) / 8 * 8 * a.mtiles);
  const int ks = a.splits / KT;
  if constexpr (KT == 1) {
    if (ks == 8) {
      hipLaunchKernelGGL((k_gemm_ks<8, 1, NT, PF, EPI, ONE>), grid, dim3(8 * 64), 0, s, a);
      return hipGetLastError();
    }
    if (ks == 4) {
      hipLaunchKernelGGL((k_gemm_ks<4, 1, NT, PF, EPI, ONE>), grid, dim3(4 * 64), 0, s, a);
      return hipGetLastError();
    }
  } else {
    if (ks == 4) {
      hipLaunchKernelGGL((k_gemm_ks<4, KT, NT, PF, EPI, ONE>), grid, dim3(4 * KT * 64), 0, s, a);
      return hipGetLastError();
    }
    if (ks == 2) {
      hipLaunchKernelGGL((k_gemm_ks<2, KT, NT, PF, EPI, ONE>), grid, dim3(2 * KT * 64), 0, s, a);
      return hipGetLastError();
    }
  }
  return hipErrorInvalidValue;
}

template <int EPI, int NT>
static hipError_t launch_nt(const GemmArgs& a, hipStream_t s) {
  const bool one = a.map == MAP_SINGLE || a.map == MAP_QKV_SINGLE;
  if constexpr (EPI == EPI_RESID || EPI == EPI_STORE || EPI == EPI_QKV_RAW) {
    if (one) return (NT == 1 && a.tgroups == 1) ? launch_one<EPI, 1, 1, true>(a, s) : hipErrorInvalidValue;
  }
  if (one) return hipErrorInvalidValue;
  if constexpr (EPI == EPI_QKV_RAW) {
    return hipErrorInvalidValue;
  } else {
    if (a.tgroups == 1) return launch_one<EPI, 1, NT, false>(a, s);
    return hipErrorInvalidValue;
  }
}

template <int EPI>
static hipError_t launch_epi(const GemmArgs& a, int NT, hipStream_t s) {
  switch (NT) {
    case 1: return launch_nt<EPI, 1>(a, s);
    case 2: return launch_nt<EPI, 2>(a, s);
    case 3: return launch_nt<EPI, 3>(a, s);
    case 4: return launch_nt<EPI, 4>(a, s);
    case 5: return launch_nt<EPI, 5>(a, s);
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
    case EPI_QKV_RAW: return launch_epi<EPI_QKV_RAW>(a, NT, s);
    case EPI_PATCH: return launch_epi<EPI_PATCH>(a, NT, s);
    case EPI_GELU: return launch_epi<EPI_GELU>(a, NT, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace gvc
