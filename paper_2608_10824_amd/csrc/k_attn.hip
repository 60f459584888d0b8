// Causal attention of the recomputed query rows over the mixed K/V cache.
//
// Alg. 1's partial forward pass recomputes only some tokens; their queries
// attend over keys of which some were just written (recomputed rows) and the
// rest are carried over from the previous frame (reused rows).  Both sit in
// the same per-layer cache, so the kernel is an ordinary causal attention
// whose queries are an arbitrary, position-sorted subset of the prompt.
//
// Prefill: one workgroup per (episode, head, 16 query rows), its waves
// splitting the key tiles.  Rows at positions >= block_first form a
// bidirectional block: they see every key up to block_last (the OFT action
// chunk decoded in parallel); block_first > block_last leaves all causal.  S = Q K^T and O += P V
// run on MFMA v_mfma_f32_16x16x32_bf16 over key tiles of 32 with an fp32
// online softmax; P is re-laid out through a 1 KiB LDS tile into the A
// operand order; V is stored transposed so the B operand of P V is 16
// contiguous bytes per lane.
// Decode: one workgroup per (head, episode) and one query.
#include "gvc_kernels.h"
#include "gvc_sync.h"

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
#define GPA(p) ((const void __attribute__((address_space(1)))*)(p))
#define LPA(p) ((void __attribute__((address_space(3)))*)(p))

namespace gvc {

// kAttnWaves waves per (episode, head, 16 query rows) split the key tiles
// round robin; each keeps its own online softmax (running max, sum and
// output), and the partial results are merged through LDS at the end.
constexpr int kAttnWaves = 4;
// Row stride (bf16) of a wave's 16 x 32 tile of probabilities in LDS.  With
// 64-byte rows the four row groups of a store and the sixteen rows of an
// operand read share banks; 80-byte rows cut the counted bank conflicts
// (38% -> 30% of the LDS cycles) but measured slower (grouped attention 70
// against 60 us per layer, 16 episodes at 50% reuse), so rows stay dense.
constexpr int kPsStride = 32;

template <int DH>
__global__ __launch_bounds__(kAttnWaves * 64) void k_attn_prefill(
    const bf16* __restrict__ q, const bf16* __restrict__ kc, const bf16* __restrict__ vc,
    const int* __restrict__ rows_pos, const int* __restrict__ ep_counts, const int* __restrict__ ep_offsets, int H,
    int kv_pad, bf16* __restrict__ o, int KB, int block_first, int block_last) {
  constexpr int NK = DH / 32;   // k-steps of QK^T
  constexpr int NO = DH / 16;   // output column blocks
  static_assert(NO % kAttnWaves == 0, "output blocks per merging wave");
  __shared__ __attribute__((aligned(16))) bf16 ps_all[kAttnWaves][16 * kPsStride];
  __shared__ floatx4 m_acc[kAttnWaves][NO][64];
  __shared__ float m_ml[kAttnWaves][8][64];
  const int tile = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int cnt = ep_counts[b];
  if (tile * 16 >= cnt) return;
  const int off = ep_offsets[b];
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  bf16* ps = ps_all[wv];
  const int col = lane & 15, grp = lane >> 4;
  const int d = H * DH;
  const int last = min(cnt, tile * 16 + 16) - 1;     // last valid row of the tile
  // last key a row at position p sees (non-decreasing in p; rows are sorted)
  auto key_last = [&](int p) { return p >= block_first ? block_last : p; };
  const int max_pos = key_last(rows_pos[off + last]);
  // this lane's rows in the C layout
  int qpos[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = min(tile * 16 + grp * 4 + i, last);
    qpos[i] = key_last(rows_pos[off + r]);
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

  // This wave's key tiles: j0 = 32 * (wv + kAttnWaves * n) <= max_pos.  Key
  // tile j0's fragments are loaded during the wave's previous tile and its
  // value fragments at the start of tile j0, so both round trips overlap the
  // arithmetic (the last tile re-reads itself instead of reading past it).
  // A row may see no key at all in a wave's tiles: its running max stays
  // -inf and the update keeps its sum and output at zero.
  constexpr int kStride = 32 * kAttnWaves;
  bf16x8 kf0[NK], kf1[NK], vf[NO];
  auto load_k = [&](int j, bf16x8 (&f0)[NK], bf16x8 (&f1)[NK]) {
    const bf16* k0 = kbase + (size_t)(j + col) * DH + grp * 8;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      f0[kk] = *(const bf16x8*)(k0 + kk * 32);
      f1[kk] = *(const bf16x8*)(k0 + 16 * DH + kk * 32);
    }
  };
  const int jstart = 32 * wv;
  if (jstart <= max_pos) load_k(jstart, kf0, kf1);
  for (int j0 = jstart; j0 <= max_pos; j0 += kStride) {
    {
      const bf16* vj = vbase + j0 + grp * 8;
#pragma unroll
      for (int c = 0; c < NO; ++c) vf[c] = *(const bf16x8*)(vj + (size_t)(c * 16 + col) * kv_pad);
    }
    bf16x8 nk0[NK], nk1[NK];
    load_k(j0 + kStride <= max_pos ? j0 + kStride : j0, nk0, nk1);
    floatx4 s0 = {0, 0, 0, 0}, s1 = {0, 0, 0, 0};
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      s0 = mfma16(qf[kk], kf0[kk], s0);
      s1 = mfma16(qf[kk], kf1[kk], s1);
    }
    float p0[4], p1[4], alpha[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float a0 = (j0 + col <= qpos[i]) ? s0[i] * scale : -INFINITY;
      const float a1 = (j0 + 16 + col <= qpos[i]) ? s1[i] * scale : -INFINITY;
      const float mx = group_max<16>(fmaxf(a0, a1));   // over the row's 16 lanes (one DPP row)
      const float mn = fmaxf(m_run[i], mx);
      const float mb = mn == -INFINITY ? 0.f : mn;      // no key yet: everything stays zero
      alpha[i] = __expf(m_run[i] - mb);
      p0[i] = __expf(a0 - mb);
      p1[i] = __expf(a1 - mb);
      const float sm = group_sum<16>(p0[i] + p1[i]);
      l_run[i] = l_run[i] * alpha[i] + sm;
      m_run[i] = mn;
    }
#pragma unroll
    for (int c = 0; c < NO; ++c)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[c][i] *= alpha[i];
    // P (C layout: row grp*4+i, key col / 16+col) -> this wave's LDS tile
    // [16][32] -> A layout (a wave's LDS accesses complete in order)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ps[(grp * 4 + i) * kPsStride + col] = f2bf(p0[i]);
      ps[(grp * 4 + i) * kPsStride + 16 + col] = f2bf(p1[i]);
    }
    const bf16x8 pa = *(const bf16x8*)(ps + col * kPsStride + grp * 8);
#pragma unroll
    for (int c = 0; c < NO; ++c) acc[c] = mfma16(pa, vf[c], acc[c]);
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      kf0[kk] = nk0[kk];
      kf1[kk] = nk1[kk];
    }
  }
  // merge the waves' partial softmax results; wave w finishes output blocks
  // [w NO / kAttnWaves, (w + 1) NO / kAttnWaves) for all 16 rows
#pragma unroll
  for (int c = 0; c < NO; ++c) m_acc[wv][c][lane] = acc[c];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    m_ml[wv][i][lane] = m_run[i];
    m_ml[wv][4 + i][lane] = l_run[i];
  }
  __syncthreads();
  float lt[4], sw[kAttnWaves][4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float m = m_ml[0][i][lane];
#pragma unroll
    for (int w = 1; w < kAttnWaves; ++w) m = fmaxf(m, m_ml[w][i][lane]);   // finite: wave 0 sees key 0
    float l = 0.f;
#pragma unroll
    for (int w = 0; w < kAttnWaves; ++w) {
      sw[w][i] = __expf(m_ml[w][i][lane] - m);
      l += m_ml[w][4 + i][lane] * sw[w][i];
    }
    lt[i] = l;
  }
  constexpr int CW = NO / kAttnWaves;
#pragma unroll
  for (int cc = 0; cc < CW; ++cc) {
    const int c = wv * CW + cc;
    floatx4 v = {0, 0, 0, 0};
#pragma unroll
    for (int w = 0; w < kAttnWaves; ++w) {
      const floatx4 aw = m_acc[w][c][lane];
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] += aw[i] * sw[w][i];
    }
    // normalise and store (frag layout for the output projection)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = tile * 16 + grp * 4 + i;
      if (r < cnt) o[frag_off(off + r, h * DH + c * 16 + col, KB)] = f2bf(v[i] / lt[i]);
    }
  }
}

// Grouped variant for many-row sessions (DH = 128): one workgroup of
// kGrpWaves waves per (episode, head, kGrpWaves query tiles of 16 rows).
// Wave w owns query tile blockIdx.x * kGrpWaves + w and walks every key tile
// up to its rows' last key with one online softmax (no merge across waves).
// Each key tile's K rows and V columns (32 keys) are copied once per
// workgroup straight into LDS (global_load_lds), three stages deep with one
// barrier per tile; a stage is overwritten two tiles after it was read, once
// every wave has passed the barrier in between.  The 16-byte chunks sit
// XOR-swizzled in LDS (K: chunk ^ key % 16 within a key row; V: chunk ^
// (dim / 4) % 4 within a dimension's 32 keys), so the 16 lanes that read one
// MFMA operand row group hit distinct banks; each lane of a copy fetches the
// global chunk that belongs at its LDS slot.  Per row the arithmetic is that
// of a single wave walking all of its key tiles in order: a tile entirely
// past a row's last key leaves its running max, sum and output unchanged, so
// a row's result does not depend on which rows share its tile.
constexpr int kGrpWaves = 4, kGrpStages = 3;
constexpr int kGrpChunks = 32 * 128 * 2 / 16;           // 16-byte chunks per K (or V) tile
constexpr int kGrpCopies = kGrpChunks / (kGrpWaves * 64);   // copies per wave per tile, each of K and V

__global__ __launch_bounds__(kGrpWaves * 64) void k_attn_prefill_grp(
    const bf16* __restrict__ q, const bf16* __restrict__ kc, const bf16* __restrict__ vc,
    const int* __restrict__ rows_pos, const int* __restrict__ ep_counts, const int* __restrict__ ep_offsets, int H,
    int kv_pad, bf16* __restrict__ o, int KB, int block_first, int block_last) {
  constexpr int DH = 128, NK = DH / 32, NO = DH / 16;
  static_assert(kGrpCopies * kGrpWaves * 64 == kGrpChunks, "tile copies");
  __shared__ u32x4 kv_lds[kGrpStages][2][kGrpChunks];
  __shared__ __attribute__((aligned(16))) bf16 ps_all[kGrpWaves][16 * kPsStride];
  const int h = blockIdx.y, b = blockIdx.z;
  const int cnt = ep_counts[b];
  const int row0 = blockIdx.x * kGrpWaves * 16;
  if (row0 >= cnt) return;   // uniform over the workgroup
  const int off = ep_offsets[b];
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  bf16* ps = ps_all[wv];
  const int col = lane & 15, grp = lane >> 4;
  const int d = H * DH;
  auto key_last = [&](int p) { return p >= block_first ? block_last : p; };
  // key tiles of the workgroup: up to the last key of its last row
  const int wg_last = min(cnt, row0 + kGrpWaves * 16) - 1;
  const int ntiles = key_last(rows_pos[off + wg_last]) / 32 + 1;
  const int tile = blockIdx.x * kGrpWaves + wv;
  const bool active = tile * 16 < cnt;
  const int last = active ? min(cnt, tile * 16 + 16) - 1 : wg_last;
  const int max_pos = active ? key_last(rows_pos[off + last]) : -1;
  int qpos[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) qpos[i] = key_last(rows_pos[off + min(tile * 16 + grp * 4 + i, last)]);
  bf16x8 qf[NK];
  {
    const int r = min(tile * 16 + col, last);
    const bf16* qr = q + (size_t)(off + r) * d + h * DH + grp * 8;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) qf[kk] = *(const bf16x8*)(qr + kk * 32);
  }
  const bf16* kbase = kc + (size_t)(b * H + h) * kv_pad * DH;
  const bf16* vbase = vc + (size_t)(b * H + h) * DH * kv_pad;
  // copy n of tile t: K slots n*64 + lane (key n*4 + lane/16, chunk lane%16),
  // V slots n*64 + lane (dimension n*16 + lane/4, chunk lane%4); tiles past
  // the last re-read it (in bounds)
  auto issue = [&](int t) {
    const int j0 = min(t, ntiles - 1) * 32;
    u32x4* st = kv_lds[t % kGrpStages][0];
#pragma unroll
    for (int c = 0; c < kGrpCopies; ++c) {
      const int n = wv * kGrpCopies + c;
      const int key = n * 4 + (lane >> 4), kch = (lane & 15) ^ (key & 15);
      __builtin_amdgcn_global_load_lds(GPA(kbase + (size_t)(j0 + key) * DH + kch * 8), LPA(st + n * 64), 16, 0, 0);
    }
#pragma unroll
    for (int c = 0; c < kGrpCopies; ++c) {
      const int n = wv * kGrpCopies + c;
      const int dim = n * 16 + (lane >> 2), vch = (lane & 3) ^ ((dim >> 2) & 3);
      __builtin_amdgcn_global_load_lds(GPA(vbase + (size_t)dim * kv_pad + j0 + vch * 8),
                                       LPA(st + kGrpChunks + n * 64), 16, 0, 0);
    }
  };
  const float scale = 1.0f / sqrtf((float)DH);
  floatx4 acc[NO];
#pragma unroll
  for (int c = 0; c < NO; ++c) acc[c] = floatx4{0, 0, 0, 0};
  float m_run[4], l_run[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) { m_run[i] = -INFINITY; l_run[i] = 0.f; }
  issue(0);
  for (int t = 0; t < ntiles; ++t) {
    issue(t + 1);
    wait_vmcnt<2 * kGrpCopies>();
    lds_barrier();
    const int j0 = t * 32;
    if (j0 > max_pos) continue;   // uniform per wave; the barrier of the next tile is still reached
    const u32x4* kt = kv_lds[t % kGrpStages][0];
    const u32x4* vt = kv_lds[t % kGrpStages][1];
    floatx4 s0 = {0, 0, 0, 0}, s1 = {0, 0, 0, 0};
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      const int ch = (kk * 4 + grp) ^ col;   // key col (and 16 + col): key % 16 == col
      s0 = mfma16(qf[kk], __builtin_bit_cast(bf16x8, kt[col * 16 + ch]), s0);
      s1 = mfma16(qf[kk], __builtin_bit_cast(bf16x8, kt[(16 + col) * 16 + ch]), s1);
    }
    float p0[4], p1[4], alpha[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float a0 = (j0 + col <= qpos[i]) ? s0[i] * scale : -INFINITY;
      const float a1 = (j0 + 16 + col <= qpos[i]) ? s1[i] * scale : -INFINITY;
      const float mx = group_max<16>(fmaxf(a0, a1));
      const float mn = fmaxf(m_run[i], mx);
      const float mb = mn == -INFINITY ? 0.f : mn;
      alpha[i] = __expf(m_run[i] - mb);
      p0[i] = __expf(a0 - mb);
      p1[i] = __expf(a1 - mb);
      const float sm = group_sum<16>(p0[i] + p1[i]);
      l_run[i] = l_run[i] * alpha[i] + sm;
      m_run[i] = mn;
    }
#pragma unroll
    for (int c = 0; c < NO; ++c)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[c][i] *= alpha[i];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ps[(grp * 4 + i) * kPsStride + col] = f2bf(p0[i]);
      ps[(grp * 4 + i) * kPsStride + 16 + col] = f2bf(p1[i]);
    }
    const bf16x8 pa = *(const bf16x8*)(ps + col * kPsStride + grp * 8);
#pragma unroll
    for (int c = 0; c < NO; ++c) {
      // dimension c*16 + col, keys grp*8..: chunk grp ^ (dim / 4) % 4 = grp ^ col / 4
      const bf16x8 vf = __builtin_bit_cast(bf16x8, vt[(c * 16 + col) * 4 + (grp ^ (col >> 2))]);
      acc[c] = mfma16(pa, vf, acc[c]);
    }
  }
  wait_vmcnt<0>();
  if (!active) return;
#pragma unroll
  for (int c = 0; c < NO; ++c)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = tile * 16 + grp * 4 + i;
      if (r < cnt) o[frag_off(off + r, h * DH + c * 16 + col, KB)] = f2bf(acc[c][i] / l_run[i]);
    }
}

// Stage 2 signal (Sec. III-B: static patches that draw the instruction's
// attention are recomputed): for head h of episode b, the exact softmax of
// each instruction token after the image (positions N+1 .. N+T1, the T1 <= 32
// text rows that follow the visual block in the position-sorted row list)
// over the keys up to its position, and per visual key n the sum of those
// probabilities over the rows, written to tv[n].  Scores on MFMA as in
// k_attn_prefill (16-row tiles, key tiles of 32 over the 4 waves, kept in
// registers); three passes: row maxima, row sums, column sums in a fixed
// order (deterministic).  Either output may be null.  ent (Stage 3): per
// head, the sum over the rows (in order) of each row's entropy divided by
// log of its key count, the entropy taken as log Z - (sum_j e_j x_j) / Z
// with x_j the max-shifted score, e_j = exp(x_j) and Z = sum_j e_j (the row
// sums of pass 2).
constexpr int kTvWaves = 4, kTvTiles = 5;   // key tiles per wave: keys < 4 * 5 * 32 = 640

template <int DH>
__global__ __launch_bounds__(kTvWaves * 64) void k_text_vis(const bf16* __restrict__ q, const bf16* __restrict__ kc,
                                                           const int* __restrict__ ep_counts,
                                                           const int* __restrict__ ep_offsets, int H, int kv_pad,
                                                           int N, int P, int T1, float* __restrict__ tv,
                                                           size_t tv_bstride, float* __restrict__ ent,
                                                           size_t ent_bstride) {
  constexpr int NK = DH / 32;
  __shared__ float red[kTvWaves][32], redx[kTvWaves][32];
  __shared__ float mrow[32], lrow[32], hrow[32];
  const int h = blockIdx.x, b = blockIdx.y;
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15, grp = lane >> 4;
  const int cnt = ep_counts[b], off = ep_offsets[b];
  const int first = cnt - (P - N - 1);   // list index of position N + 1
  const int d = H * DH;
  const int nkeys = N + T1 + 1, ntile = (nkeys + 31) / 32;
  const float scale = 1.0f / sqrtf((float)DH);
  bf16x8 qf[2][NK];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const int r = min(rt * 16 + col, T1 - 1);
    const bf16* qr = q + (size_t)(off + first + r) * d + h * DH + grp * 8;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) qf[rt][kk] = *(const bf16x8*)(qr + kk * 32);
  }
  const bf16* kbase = kc + (size_t)(b * H + h) * kv_pad * DH;
  floatx4 sc[kTvTiles][2][2];   // [tile of this wave][row tile][key half]
#pragma unroll
  for (int m = 0; m < kTvTiles; ++m) {
    const int t = wv + kTvWaves * m;
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) sc[m][rt][0] = sc[m][rt][1] = floatx4{0, 0, 0, 0};
    if (t < ntile) {
      const bf16* k0 = kbase + (size_t)(32 * t + col) * DH + grp * 8;
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) {
        const bf16x8 kf0 = *(const bf16x8*)(k0 + kk * 32), kf1 = *(const bf16x8*)(k0 + 16 * DH + kk * 32);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          sc[m][rt][0] = mfma16(qf[rt][kk], kf0, sc[m][rt][0]);
          sc[m][rt][1] = mfma16(qf[rt][kk], kf1, sc[m][rt][1]);
        }
      }
    }
  }
  // row r = rt * 16 + grp * 4 + i sees key j when r < T1 and j <= N + 1 + r
  auto seen = [&](int m, int rt, int hf, int i) {
    const int t = wv + kTvWaves * m, r = rt * 16 + grp * 4 + i, j = 32 * t + 16 * hf + col;
    return t < ntile && r < T1 && j <= N + 1 + r;
  };
  // pass 1: row maxima
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mx = -INFINITY;
#pragma unroll
      for (int m = 0; m < kTvTiles; ++m)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
          if (seen(m, rt, hf, i)) mx = fmaxf(mx, sc[m][rt][hf][i] * scale);
      mx = group_max<16>(mx);
      if (col == 0) red[wv][rt * 16 + grp * 4 + i] = mx;
    }
  __syncthreads();
  if (threadIdx.x < 32) {
    float mx = red[0][threadIdx.x];
#pragma unroll
    for (int w = 1; w < kTvWaves; ++w) mx = fmaxf(mx, red[w][threadIdx.x]);
    mrow[threadIdx.x] = mx;
  }
  __syncthreads();
  // pass 2: row sums
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = rt * 16 + grp * 4 + i;
      const float mr = mrow[min(r, 31)];
      float sm = 0.f, sx = 0.f;
#pragma unroll
      for (int m = 0; m < kTvTiles; ++m)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
          if (seen(m, rt, hf, i)) {
            const float x = sc[m][rt][hf][i] * scale - mr, e = __expf(x);
            sm += e;
            sx += e * x;
          }
      sm = group_sum<16>(sm);
      if (col == 0) red[wv][r] = sm;
      if (ent) {
        sx = group_sum<16>(sx);
        if (col == 0) redx[wv][r] = sx;
      }
    }
  __syncthreads();
  if (threadIdx.x < 32) {
    float sm = 0.f, sx = 0.f;
#pragma unroll
    for (int w = 0; w < kTvWaves; ++w) {
      sm += red[w][threadIdx.x];
      sx += ent ? redx[w][threadIdx.x] : 0.f;
    }
    lrow[threadIdx.x] = sm;
    const int r = threadIdx.x;
    hrow[r] = r < T1 ? (__logf(sm) - sx / sm) / __logf((float)(N + 2 + r)) : 0.f;
  }
  __syncthreads();
  if (ent && threadIdx.x == 0) {
    float e = 0.f;
    for (int r = 0; r < T1; ++r) e += hrow[r];
    ent[(size_t)b * ent_bstride + h] = e;
  }
  if (!tv) return;
  // pass 3: per visual key (1 <= j <= N) the sum of the rows' probabilities
  float* out = tv + (size_t)b * tv_bstride + (size_t)h * N;
#pragma unroll
  for (int m = 0; m < kTvTiles; ++m)
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int t = wv + kTvWaves * m, j = 32 * t + 16 * hf + col;
      float cs = 0.f;
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = rt * 16 + grp * 4 + i;
          if (seen(m, rt, hf, i)) cs += __expf(sc[m][rt][hf][i] * scale - mrow[r]) / lrow[r];
        }
      cs += __shfl_xor(cs, 16);
      cs += __shfl_xor(cs, 32);
      if (grp == 0 && t < ntile && j >= 1 && j <= N) out[j - 1] = cs;
    }
}

// Single-query attention of a decode pass at position pos.  One workgroup
// per (head, episode, value slice): q and the new key arrive un-rotated in
// fp32; every workgroup rotates them (RoPE, pairing dim i with i + DH/2), the
// first slice also stores the rotated key (bf16) into the cache, and each
// computes all pos + 1 scores but only its DH/NQ value dimensions, so a head
// spreads over NQ workgroups without any cross-workgroup combine.
// The first batch of key rows and the value runs are loaded before anything
// else, so their latency overlaps the rotation; longer sequences loop.
// Scores: DH/8 lanes per key, each a 16-byte run of dims (a wave instruction
// reads whole key rows); the new key comes from LDS, never from the cache
// slot being written.  Values: the cache is dim-major, so a lane reads 8
// consecutive keys of one dim.
template <int DH, int NQ>
__global__ __launch_bounds__(512, 4) void k_attn_decode(const float* __restrict__ qraw, const float* __restrict__ kraw,
                                                     bf16* __restrict__ kc, const bf16* __restrict__ vc,
                                                     const float2* __restrict__ rope, int H, int kv_pad, int pos,
                                                     bf16* __restrict__ o, int KB) {
  extern __shared__ float sc[];          // [kv_pad] scores, then probabilities
  __shared__ float qs[DH], kn[DH];
  __shared__ float red[16];
  constexpr int NT = 512;
  constexpr int LPK = DH / 8;            // lanes per key
  constexpr int KPI = NT / LPK;          // keys per load round
  constexpr int U = 9;                   // load rounds per batch
  constexpr int DQ = DH / NQ;            // value dims of this workgroup
  constexpr int DG = NT / 16;            // dim groups
  constexpr int ND = (DQ + DG - 1) / DG; // dims per thread in the value phase
  constexpr int UC = 2;                  // 8-key chunks per lane per value batch
  const int h = blockIdx.x, b = blockIdx.y, qd = blockIdx.z;
  const int d = H * DH, half = DH / 2;
  const int tid = threadIdx.x;
  const int n_keys = pos + 1;
  const int nchunk = (n_keys + 7) / 8;
  bf16* kbase = kc + (size_t)(b * H + h) * kv_pad * DH;
  const int sub = tid % LPK, kg = tid / LPK;
  const bf16* ksub = kbase + sub * 8;
  const int last_cached = max(pos - 1, 0);
  // value-phase mapping: lane16 walks 8-key chunks, DG dim groups
  const int l16 = tid & 15, dg = tid >> 4;
  const bf16* vb = vc + (size_t)(b * H + h) * DH * kv_pad + (size_t)(qd * DQ) * kv_pad;
  u16x8 kv[U], vv[ND][UC];
#pragma unroll
  for (int u = 0; u < U; ++u) kv[u] = *(const u16x8*)(ksub + (size_t)min(u * KPI + kg, last_cached) * DH);
#pragma unroll
  for (int i = 0; i < ND; ++i)
#pragma unroll
    for (int u = 0; u < UC; ++u)
      vv[i][u] = *(const u16x8*)(vb + (size_t)min(dg + DG * i, DQ - 1) * kv_pad + min(16 * u + l16, nchunk - 1) * 8);
  if (tid < half) {
    const float2 cs = rope[(size_t)pos * half + tid];
    const float* qr = qraw + (size_t)b * d + h * DH;
    const float* kr = kraw + (size_t)b * d + h * DH;
    const float q0 = qr[tid], q1 = qr[tid + half], k0 = kr[tid], k1 = kr[tid + half];
    qs[tid] = q0 * cs.x - q1 * cs.y;
    qs[tid + half] = q1 * cs.x + q0 * cs.y;
    const bf16 ka = f2bf(k0 * cs.x - k1 * cs.y), kb = f2bf(k1 * cs.x + k0 * cs.y);
    kn[tid] = bf2f(ka);
    kn[tid + half] = bf2f(kb);
    if (qd == 0) {
      kbase[(size_t)pos * DH + tid] = ka;
      kbase[(size_t)pos * DH + tid + half] = kb;
    }
  }
  __syncthreads();
  float qv[8], kv_new[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) { qv[i] = qs[sub * 8 + i]; kv_new[i] = kn[sub * 8 + i]; }
  const float scale = 1.0f / sqrtf((float)DH);
  float mx = -INFINITY;
  for (int j0 = 0; j0 < n_keys; j0 += KPI * U) {
    if (j0 > 0) {
#pragma unroll
      for (int u = 0; u < U; ++u) kv[u] = *(const u16x8*)(ksub + (size_t)min(j0 + u * KPI + kg, last_cached) * DH);
    }
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
  mx = red[0];
#pragma unroll
  for (int w = 1; w < NT / 64; ++w) mx = fmaxf(mx, red[w]);
  float sm = 0.f;
  for (int j = tid; j < n_keys; j += NT) {
    const float p = __expf(sc[j] - mx);
    sc[j] = p;
    sm += p;
  }
  for (int x = 32; x > 0; x >>= 1) sm += __shfl_xor(sm, x);
  __syncthreads();
  if ((tid & 63) == 0) red[8 + (tid >> 6)] = sm;
  for (int j = n_keys + tid; j < nchunk * 8; j += NT) sc[j] = 0.f;   // pad the last 8-key chunk
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) tot += red[8 + w];
  const float inv = 1.0f / tot;
  float acc[ND];
#pragma unroll
  for (int i = 0; i < ND; ++i) acc[i] = 0.f;
  for (int c0 = 0; c0 < nchunk; c0 += 16 * UC) {
    if (c0 > 0) {
#pragma unroll
      for (int i = 0; i < ND; ++i)
#pragma unroll
        for (int u = 0; u < UC; ++u)
          vv[i][u] = *(const u16x8*)(vb + (size_t)min(dg + DG * i, DQ - 1) * kv_pad +
                                     min(c0 + 16 * u + l16, nchunk - 1) * 8);
    }
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
    const int dim = dg + DG * i;
    if (l16 == 0 && dim < DQ) o[frag_off(b, h * DH + qd * DQ + dim, KB)] = f2bf(t * inv);
  }
}

hipError_t launch_attn_prefill(const bf16* q, const bf16* kc, const bf16* vc, const int* rows_pos,
                               const int* ep_counts, const int* ep_offsets, int B, int H, int head_dim, int kv_pad,
                               int max_tiles, bf16* o, int KB, int block_first, int block_last, bool grouped,
                               hipStream_t s) {
  if (block_first <= block_last && block_last >= kv_pad) return hipErrorInvalidValue;
  if (grouped && head_dim == 128) {
    const dim3 grid_g((max_tiles + kGrpWaves - 1) / kGrpWaves, H, B);
    hipLaunchKernelGGL(k_attn_prefill_grp, grid_g, dim3(kGrpWaves * 64), 0, s, q, kc, vc, rows_pos, ep_counts,
                       ep_offsets, H, kv_pad, o, KB, block_first, block_last);
    return hipGetLastError();
  }
  dim3 grid(max_tiles, H, B);
  if (head_dim == 128)
    hipLaunchKernelGGL(k_attn_prefill<128>, grid, dim3(kAttnWaves * 64), 0, s, q, kc, vc, rows_pos, ep_counts,
                       ep_offsets, H, kv_pad, o, KB, block_first, block_last);
  else if (head_dim == 64)
    hipLaunchKernelGGL(k_attn_prefill<64>, grid, dim3(kAttnWaves * 64), 0, s, q, kc, vc, rows_pos, ep_counts,
                       ep_offsets, H, kv_pad, o, KB, block_first, block_last);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_text_vis(const bf16* q, const bf16* kc, const int* ep_counts, const int* ep_offsets, int B, int H,
                           int head_dim, int kv_pad, int N, int P, int T1, float* tv, size_t tv_bstride,
                           float* ent, size_t ent_bstride, hipStream_t s) {
  if (T1 < 1 || T1 > 32 || N + T1 + 1 > kTvWaves * kTvTiles * 32 || (!tv && !ent)) return hipErrorInvalidValue;
  const dim3 grid(H, B);
  if (head_dim == 128)
    hipLaunchKernelGGL(k_text_vis<128>, grid, dim3(kTvWaves * 64), 0, s, q, kc, ep_counts, ep_offsets, H, kv_pad, N,
                       P, T1, tv, tv_bstride, ent, ent_bstride);
  else if (head_dim == 64)
    hipLaunchKernelGGL(k_text_vis<64>, grid, dim3(kTvWaves * 64), 0, s, q, kc, ep_counts, ep_offsets, H, kv_pad, N,
                       P, T1, tv, tv_bstride, ent, ent_bstride);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attn_decode(const float* qraw, const float* kraw, bf16* kc, const bf16* vc, const float2* rope,
                              int B, int H, int head_dim, int kv_pad, int pos, bf16* o, int KB, hipStream_t s) {
  const size_t shm = (size_t)kv_pad * sizeof(float);
  // Value slices per (head, episode): 4 when there are few (head, episode)
  // pairs, so the grid still covers the chip; 1 once there are 256 or more,
  // so the keys are read once (each slice recomputes every score).  The
  // arithmetic of every output is the same either way.
  const bool one = B * H >= 256;
  if (head_dim == 128 && one)
    hipLaunchKernelGGL((k_attn_decode<128, 1>), dim3(H, B, 1), dim3(512), shm, s, qraw, kraw, kc, vc, rope, H, kv_pad,
                       pos, o, KB);
  else if (head_dim == 128)
    hipLaunchKernelGGL((k_attn_decode<128, 4>), dim3(H, B, 4), dim3(512), shm, s, qraw, kraw, kc, vc, rope, H, kv_pad,
                       pos, o, KB);
  else if (head_dim == 64 && one)
    hipLaunchKernelGGL((k_attn_decode<64, 1>), dim3(H, B, 1), dim3(512), shm, s, qraw, kraw, kc, vc, rope, H, kv_pad,
                       pos, o, KB);
  else if (head_dim == 64)
    hipLaunchKernelGGL((k_attn_decode<64, 4>), dim3(H, B, 4), dim3(512), shm, s, qraw, kraw, kc, vc, rope, H, kv_pad,
                       pos, o, KB);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace gvc
