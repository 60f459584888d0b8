// Stage 1 static-patch detection and the applied per-layer reuse proportion.
//
// Sec. III-B, Stage 1: corresponding p x p patches of I_t and I_{t-1} are
// compared by cosine similarity; similarity above tau marks a patch static.
// Stage 3 (applied): each layer reuses its own share of the static set.
// Everything is integer: per patch the exact dot product and both squared
// norms (int32: 588 * 255^2 < 2^31), the test dot^2 den^2 > num^2 na nb and
// the ranking comparator dot_i^2 na_j nb_j vs dot_j^2 na_i nb_i in 128-bit
// unsigned arithmetic, so the masks are exact.
#include "gvc_kernels.h"

#include <mutex>
#include <vector>

namespace gvc {

// Patch statistics of the allocation-free selection (select_scratch): the
// [B][N][3] int32 buffer between k_patch_stats and k_rank_mask for at most
// kSelectScratchEpisodes episodes of kSelectScratchPatches patches.  Each GPU
// the library runs on holds its own copy until the process ends.
static __device__ __align__(256) int scratch[kSelectScratchEpisodes * kSelectScratchPatches * 3];

// One wave per patch: stats[(b*N + n)*3 + {0,1,2}] = dot, |u|^2, |v|^2.
__global__ __launch_bounds__(64) void k_patch_stats(const uint8_t* __restrict__ ft, const uint8_t* __restrict__ fp,
                                                    int views, int img, int patch, int* __restrict__ stats) {
  const int n = blockIdx.x, b = blockIdx.y;
  const int side = img / patch, per_view = side * side;
  const int v = n / per_view, rc = n % per_view, r = rc / side, c = rc % side;
  const int row_bytes = patch * 3;
  const size_t frame_bytes = (size_t)views * img * img * 3;
  const size_t base = (size_t)b * frame_bytes + ((size_t)v * img * img + (size_t)r * patch * img + (size_t)c * patch) * 3;
  int dot = 0, na = 0, nb = 0;
  for (int e = threadIdx.x; e < patch * row_bytes; e += 64) {
    const int pr = e / row_bytes, pc = e % row_bytes;
    const size_t off = base + (size_t)pr * img * 3 + pc;
    const int u = ft[off], w = fp[off];
    dot += u * w; na += u * u; nb += w * w;
  }
  for (int o = 32; o > 0; o >>= 1) {
    dot += __shfl_down(dot, o);
    na += __shfl_down(na, o);
    nb += __shfl_down(nb, o);
  }
  if (threadIdx.x == 0) {
    int* s = stats + ((size_t)b * gridDim.x + n) * 3;
    s[0] = dot; s[1] = na; s[2] = nb;
  }
}

typedef unsigned __int128 u128;

struct Permille { int q[128]; };

// One workgroup per episode: static flags, exact ranks, |S|, per-layer masks.
// With tv (Stage 2), the topk patches of highest score (sum of the LH
// columns of tv, in order; ties to the lower index) are not static.
// With ent (Stage 3, [B][L][H] per-head entropy sums over n_instr tokens),
// the per-layer proportions come from the episode's entropy: E_l = (sum over
// heads in order) / (H n_instr), u_l = 1 - E_l, s_0 = u_0,
// s_l = s_{l-1} + (u_l - s_{l-1}) * 0.5, q_l = floor(1000 clamp(s_l, 0, 1)),
// in fp32 and written to q_out [B][L]; otherwise they are pm.
__global__ __launch_bounds__(512) void k_rank_mask(const int* __restrict__ stats, int N, int L, long long tau_num,
                                                   long long tau_den, Permille pm, uint8_t* __restrict__ mask,
                                                   int* __restrict__ n_static, const float* __restrict__ tv, int LH,
                                                   int topk, const float* __restrict__ ent, int H, int n_instr,
                                                   int* __restrict__ q_out) {
  extern __shared__ unsigned long long sh[];   // [N] cos^2 numerator, [N] denominator (0 = not static), [N] score
  unsigned long long* knum = sh;
  unsigned long long* kden = sh + N;
  float* score = reinterpret_cast<float*>(sh + 2 * N);
  __shared__ int s_count;
  __shared__ int qs[128];
  const int b = blockIdx.x;
  if (threadIdx.x == 0) {
    s_count = 0;
    float sl = 0.f;
    for (int l = 0; l < L; ++l) {
      if (ent) {
        float e = 0.f;
        for (int h = 0; h < H; ++h) e += ent[((size_t)b * L + l) * H + h];
        const float u = 1.0f - e / (float)(H * n_instr);
        sl = l == 0 ? u : sl + (u - sl) * 0.5f;
        qs[l] = (int)floorf(1000.0f * fminf(fmaxf(sl, 0.f), 1.f));
        q_out[(size_t)b * L + l] = qs[l];
      } else {
        qs[l] = pm.q[l];
      }
    }
  }
  if (tv)
    for (int n = threadIdx.x; n < N; n += blockDim.x) {
      float sc = 0.f;
      for (int c = 0; c < LH; ++c) sc += tv[((size_t)b * LH + c) * N + n];
      score[n] = sc;
    }
  __syncthreads();
  const unsigned long long num2 = (unsigned long long)(tau_num * tau_num);
  const unsigned long long den2 = (unsigned long long)(tau_den * tau_den);
  for (int n = threadIdx.x; n < N; n += blockDim.x) {
    const int* s = stats + ((size_t)b * N + n) * 3;
    const long long dot = s[0], na = s[1], nb = s[2];
    unsigned long long kn = 0, kd = 0;   // kd == 0 marks "not static"
    if (na == 0 && nb == 0) {
      kn = 1; kd = 1;
    } else if (na != 0 && nb != 0 && dot > 0) {
      const unsigned long long d2 = (unsigned long long)dot * (unsigned long long)dot;
      const unsigned long long nn = (unsigned long long)na * (unsigned long long)nb;
      if ((u128)d2 * den2 > (u128)nn * num2) { kn = d2; kd = nn; }
    }
    if (kd && tv) {   // Stage 2: a task-relevant patch is recomputed
      const float sn = score[n];
      int above = 0;
      for (int j = 0; j < N; ++j) above += score[j] > sn || (score[j] == sn && j < n);
      if (above < topk) kd = 0;
    }
    knum[n] = kn; kden[n] = kd;
    if (kd) atomicAdd(&s_count, 1);
  }
  __syncthreads();
  const int S = s_count;
  for (int n = threadIdx.x; n < N; n += blockDim.x) {
    const unsigned long long kn = knum[n], kd = kden[n];
    int rank = 0;
    if (kd) {
      for (int j = 0; j < N; ++j) {
        const unsigned long long jd = kden[j];
        if (!jd || j == n) continue;
        const u128 lhs = (u128)knum[j] * kd, rhs = (u128)kn * jd;   // cos_j^2 vs cos_n^2
        rank += (lhs > rhs) || (lhs == rhs && j < n);
      }
    }
    for (int l = 0; l < L; ++l) {
      const int k = (int)(((long long)qs[l] * S) / 1000);
      mask[((size_t)b * L + l) * N + n] = (kd && rank < k) ? 1 : 0;
    }
  }
  if (threadIdx.x == 0 && n_static) n_static[b] = S;
}

// Device address of this GPU's copy of `scratch`, looked up once per device
// with hipGetSymbolAddress while that device is current (the array's name is
// a host-side stand-in and must never reach a kernel).
hipError_t select_scratch(int** out) {
  static std::mutex mu;
  static std::vector<int*> ptrs;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  if ((int)ptrs.size() <= dev) ptrs.resize(dev + 1, nullptr);
  if (!ptrs[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    ptrs[dev] = static_cast<int*>(p);
  }
  *out = ptrs[dev];
  return hipSuccess;
}

hipError_t launch_patch_stats(const uint8_t* ft, const uint8_t* fp, int B, int views, int img, int patch,
                              int* stats, hipStream_t s) {
  const int side = img / patch;
  dim3 grid(views * side * side, B);
  hipLaunchKernelGGL(k_patch_stats, grid, dim3(64), 0, s, ft, fp, views, img, patch, stats);
  return hipGetLastError();
}

hipError_t launch_rank_mask(const int* stats, int B, int N, int L, long long tau_num, long long tau_den,
                            const int* permille_host, uint8_t* mask, int* n_static, const float* tv, int LH,
                            int topk, const float* ent, int H, int n_instr, int* q_out, hipStream_t s) {
  if (L > 128 || (ent && (!q_out || H < 1 || n_instr < 1))) return hipErrorInvalidValue;
  Permille pm;
  for (int l = 0; l < 128; ++l) pm.q[l] = l < L ? permille_host[l] : 0;
  const size_t shm = (size_t)N * 2 * sizeof(unsigned long long) + (size_t)N * sizeof(float);
  hipLaunchKernelGGL(k_rank_mask, dim3(B), dim3(512), shm, s, stats, N, L, tau_num, tau_den, pm, mask, n_static, tv,
                     LH, topk, ent, H, n_instr, q_out);
  return hipGetLastError();
}

}  // namespace gvc
