// Backward of the chunk attention (the SDPA of a fine-tuning step, Sec.
// "Fine-Tuning for Sparse Attention"): gradients of q, k and v for the loss
// sum(dout * out), given the forward's lse. The summed weights carry no
// gradient. Float32 arithmetic on the VALU for float32 or bf16 data.
//
// With P = softmax(A), A = scale Q K^T masked, dP = dout V^T and
// D_r = sum_j P_rj dP_rj:
//   dV_j = sum_r P_rj dout_r
//   dS_rj = P_rj (dP_rj - D_r)          (softmax vector-Jacobian product)
//   dQ_r = scale sum_j dS_rj K_j,   dK_j = scale sum_r dS_rj Q_r
// summed over the G query heads of a KV head for dK and dV.
//
// D_r is taken from P and dP themselves, not from the stored output: where a
// row's weights are nearly one-hot, dS is a small difference of large terms,
// and <dout_r, out_r> with out rounded to bf16 would leave an error of the
// size of the result.
//
//   dq      block = 32 packed rows; one sweep over the key tiles the rows can
//           see accumulates sum_j P dP K_j, sum_j P K_j and D_r, then
//           dQ_r = scale (sum_j P dP K_j - D_r sum_j P K_j); D_r is stored
//   dkdv    block = 32 key columns of one KV head; loops over the head's packed
//           rows 32 at a time: P and P dP of the 32 x 32 pairs in LDS, then
//           each thread adds its (key, feature) outputs of dK and dV
//
// Keys are [cache || chunk] (chunk mode) or the cache alone with the
// token-position mask (cache mode), as in the forward kernels.
#include "internal.h"

namespace h2o {
namespace {

constexpr int kBT = 256;   // threads per block
constexpr int kKT = 32;    // keys per tile
constexpr int kRT = 32;    // packed rows per tile

struct BwdGeo {
  int Hq, Hkv, G, T, M, Tk, R, Nk;
  KeyPos kp;
};

template <typename E>
__device__ __forceinline__ const E* key_row(const E* cache, const E* fresh, size_t bh, int j,
                                            int M, int T, int d) {
  return j < M ? cache + (bh * M + j) * (size_t)d : fresh + (bh * T + (j - M)) * (size_t)d;
}

__device__ __forceinline__ bool key_visible(const BwdGeo& g, const int32_t* tp, int j, int i) {
  if (j >= g.M) return j - g.M <= i;
  return !tp || pos_visible(tp[j], g.kp.pos0, i);
}

// Row r of head bh as (query head hq, chunk position i) and its offset in
// [B,Hq,T,d] / [B,Hq,T].
__device__ __forceinline__ size_t row_index(const BwdGeo& g, size_t bh, int r) {
  const int b = (int)(bh / g.Hkv), h = (int)(bh % g.Hkv);
  const int i = r / g.G, gg = r % g.G;
  return (size_t)(b * g.Hq + h * g.G + gg) * g.T + i;
}

// P and P*dP of the pairs (rows [r0, r0+kRT), keys [j0, j0+kKT)) into ps/pd
// ([kRT][kKT+1]); Qs, dOs ([kRT][D+1]), Ks, Vs ([kKT][D+1]) staged in LDS,
// lse per row (natural log, -inf for a row that sees nothing).
template <int D>
__device__ __forceinline__ void pair_tile(const BwdGeo& g, const int32_t* tp, int r0, int j0,
                                          const float* Qs, const float* dOs, const float* Ks,
                                          const float* Vs, const float* lse_s, float scale,
                                          float* ps, float* pd) {
  for (int e = threadIdx.x; e < kRT * kKT; e += kBT) {
    const int rr = e / kKT, jj = e % kKT;
    const int r = r0 + rr, j = j0 + jj;
    float p = 0.f, pdv = 0.f;
    if (r < g.R && j < g.Nk && lse_s[rr] > -INFINITY && key_visible(g, tp, j, r / g.G)) {
      float s = 0.f, dp = 0.f;
      for (int c = 0; c < D; ++c) {
        s = fmaf(Qs[rr * (D + 1) + c], Ks[jj * (D + 1) + c], s);
        dp = fmaf(dOs[rr * (D + 1) + c], Vs[jj * (D + 1) + c], dp);
      }
      p = expf(s * scale - lse_s[rr]);
      pdv = p * dp;
    }
    ps[rr * (kKT + 1) + jj] = p;
    pd[rr * (kKT + 1) + jj] = pdv;
  }
}

// Rows [r0, r0+kRT) of head bh: q, dout, lse and, when dot is non-null, D_r.
template <typename E, int D>
__device__ __forceinline__ void stage_rows(const BwdGeo& g, size_t bh, int r0, const E* q,
                                           const E* dout, const float* lse, const float* dot,
                                           float* Qs, float* dOs, float* lse_s, float* dot_s) {
  for (int e = threadIdx.x; e < kRT * D; e += kBT) {
    const int rr = e / D, c = e % D, r = r0 + rr;
    float qv = 0.f, dv = 0.f;
    if (r < g.R) {
      const size_t o = row_index(g, bh, r) * D + c;
      qv = load_elem(q, o);
      dv = load_elem(dout, o);
    }
    Qs[rr * (D + 1) + c] = qv;
    dOs[rr * (D + 1) + c] = dv;
  }
  for (int rr = threadIdx.x; rr < kRT; rr += kBT) {
    const int r = r0 + rr;
    lse_s[rr] = r < g.R ? lse[row_index(g, bh, r)] : -INFINITY;
    if (dot) dot_s[rr] = r < g.R ? dot[bh * g.R + r] : 0.f;
  }
}

template <typename E, int D>
__device__ __forceinline__ void stage_keys(const BwdGeo& g, size_t bh, int j0, const E* kc,
                                           const E* vc, const E* kn, const E* vn, float* Ks,
                                           float* Vs) {
  for (int e = threadIdx.x; e < kKT * D; e += kBT) {
    const int jj = e / D, c = e % D, j = j0 + jj;
    float kv = 0.f, vv = 0.f;
    if (j < g.Nk) {
      kv = load_elem(key_row(kc, kn, bh, j, g.M, g.T, D), c);
      vv = load_elem(key_row(vc, vn, bh, j, g.M, g.T, D), c);
    }
    Ks[jj * (D + 1) + c] = kv;
    Vs[jj * (D + 1) + c] = vv;
  }
}

// First packed row that may see key column j (chunk key j - M: position
// j - M; cache mode and cache slots: row 0).
__device__ __forceinline__ int first_row(const BwdGeo& g, int j) {
  if (g.kp.tp || j < g.M) return 0;
  return (j - g.M) * g.G;
}

template <typename E, int D>
__global__ __launch_bounds__(kBT) void bwd_dkdv(BwdGeo g, const E* __restrict__ q,
                                                const E* __restrict__ kc,
                                                const E* __restrict__ vc,
                                                const E* __restrict__ kn,
                                                const E* __restrict__ vn,
                                                const E* __restrict__ dout,
                                                const float* __restrict__ lse,
                                                const float* __restrict__ dot, float scale,
                                                E* __restrict__ dkc, E* __restrict__ dvc,
                                                E* __restrict__ dkn, E* __restrict__ dvn) {
  constexpr int PER = kKT * D / kBT;   // (key, feature) outputs per thread
  __shared__ float Ks[kKT * (D + 1)], Vs[kKT * (D + 1)];
  __shared__ float Qs[kRT * (D + 1)], dOs[kRT * (D + 1)];
  __shared__ float ps[kRT * (kKT + 1)], pd[kRT * (kKT + 1)];
  __shared__ float lse_s[kRT], dot_s[kRT];
  const size_t bh = blockIdx.y;
  const int j0 = blockIdx.x * kKT;
  const int32_t* tp = g.kp.tp ? g.kp.tp + bh * (size_t)g.M : nullptr;
  stage_keys<E, D>(g, bh, j0, kc, vc, kn, vn, Ks, Vs);
  float dk[PER], dv[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) dk[u] = dv[u] = 0.f;
  // rows that see no key of this tile are skipped (their pairs are all 0)
  const int rstart = (first_row(g, j0) / kRT) * kRT;
  for (int r0 = rstart; r0 < g.R; r0 += kRT) {
    __syncthreads();
    stage_rows<E, D>(g, bh, r0, q, dout, lse, dot, Qs, dOs, lse_s, dot_s);
    __syncthreads();
    pair_tile<D>(g, tp, r0, j0, Qs, dOs, Ks, Vs, lse_s, scale, ps, pd);
    __syncthreads();
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = threadIdx.x + u * kBT, jj = e / D, c = e % D;
      float a = dk[u], b = dv[u];
      for (int rr = 0; rr < kRT; ++rr) {
        const float p = ps[rr * (kKT + 1) + jj];
        const float dsv = fmaf(-p, dot_s[rr], pd[rr * (kKT + 1) + jj]);   // P (dP - D)
        a = fmaf(dsv, Qs[rr * (D + 1) + c], a);
        b = fmaf(p, dOs[rr * (D + 1) + c], b);
      }
      dk[u] = a;
      dv[u] = b;
    }
  }
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = threadIdx.x + u * kBT, jj = e / D, c = e % D, j = j0 + jj;
    if (j >= g.Nk) continue;
    if (j < g.M) {
      store_elem(dkc, (bh * g.M + j) * (size_t)D + c, dk[u] * scale);
      store_elem(dvc, (bh * g.M + j) * (size_t)D + c, dv[u]);
    } else {
      store_elem(dkn, (bh * g.T + (j - g.M)) * (size_t)D + c, dk[u] * scale);
      store_elem(dvn, (bh * g.T + (j - g.M)) * (size_t)D + c, dv[u]);
    }
  }
}

template <typename E, int D>
__global__ __launch_bounds__(kBT) void bwd_dq(BwdGeo g, const E* __restrict__ q,
                                              const E* __restrict__ kc, const E* __restrict__ vc,
                                              const E* __restrict__ kn, const E* __restrict__ vn,
                                              const E* __restrict__ dout,
                                              const float* __restrict__ lse, float scale,
                                              E* __restrict__ dq, float* __restrict__ dot) {
  constexpr int PER = kRT * D / kBT;   // (row, feature) outputs per thread
  __shared__ float Ks[kKT * (D + 1)], Vs[kKT * (D + 1)];
  __shared__ float Qs[kRT * (D + 1)], dOs[kRT * (D + 1)];
  __shared__ float ps[kRT * (kKT + 1)], pd[kRT * (kKT + 1)];
  __shared__ float lse_s[kRT];
  const size_t bh = blockIdx.y;
  const int r0 = blockIdx.x * kRT;
  const int32_t* tp = g.kp.tp ? g.kp.tp + bh * (size_t)g.M : nullptr;
  stage_rows<E, D>(g, bh, r0, q, dout, lse, nullptr, Qs, dOs, lse_s, nullptr);
  float apdk[PER], apk[PER], drow[PER];   // sum P dP K, sum P K, D of the output's row
#pragma unroll
  for (int u = 0; u < PER; ++u) apdk[u] = apk[u] = drow[u] = 0.f;
  const int kv_end = kv_end_for_rows(min(r0 + kRT, g.R), g.G, g.T, g.M, g.Tk);
  for (int j0 = 0; j0 < kv_end; j0 += kKT) {
    __syncthreads();
    stage_keys<E, D>(g, bh, j0, kc, vc, kn, vn, Ks, Vs);
    __syncthreads();
    pair_tile<D>(g, tp, r0, j0, Qs, dOs, Ks, Vs, lse_s, scale, ps, pd);
    __syncthreads();
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = threadIdx.x + u * kBT, rr = e / D, c = e % D;
      float a = apdk[u], b = apk[u], dd = drow[u];
      for (int jj = 0; jj < kKT; ++jj) {
        const float kv = Ks[jj * (D + 1) + c], pdv = pd[rr * (kKT + 1) + jj];
        a = fmaf(pdv, kv, a);
        b = fmaf(ps[rr * (kKT + 1) + jj], kv, b);
        dd += pdv;
      }
      apdk[u] = a;
      apk[u] = b;
      drow[u] = dd;
    }
  }
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = threadIdx.x + u * kBT, rr = e / D, c = e % D, r = r0 + rr;
    if (r >= g.R) continue;
    store_elem(dq, row_index(g, bh, r) * D + c, scale * fmaf(-drow[u], apk[u], apdk[u]));
    if (c == 0) dot[bh * g.R + r] = drow[u];
  }
}

template <typename E, int D>
hipError_t run(const Shape& s, const void* q, const void* kc, const void* vc, const void* kn,
               const void* vn, KeyPos kp, const float* lse, const void* dout, void* dq,
               void* dkc, void* dvc, void* dkn, void* dvn, float* dot, float scale,
               hipStream_t st) {
  const BwdGeo g{s.Hq, s.Hkv, s.G(), s.T, s.M, s.Tk(), s.R(), s.Nk(), kp};
  const int BH = s.BH();
  // dq first: it leaves D_r in dot for the dk/dv kernel
  hipError_t e = launch_kernel(K_BWD_DQ, bwd_dq<E, D>, dim3((g.R + kRT - 1) / kRT, BH),
                               dim3(kBT), st, g, (const E*)q, (const E*)kc, (const E*)vc,
                               (const E*)kn, (const E*)vn, (const E*)dout, lse, scale, (E*)dq,
                               dot);
  if (e != hipSuccess || g.Nk == 0) return e;
  return launch_kernel(K_BWD_DKDV, bwd_dkdv<E, D>, dim3((g.Nk + kKT - 1) / kKT, BH), dim3(kBT),
                       st, g, (const E*)q, (const E*)kc, (const E*)vc, (const E*)kn,
                       (const E*)vn, (const E*)dout, lse, (const float*)dot, scale, (E*)dkc,
                       (E*)dvc, (E*)dkn, (E*)dvn);
}

// delta[row, i, :] = cache[row, idx[row, i], :] (gather) or
// cache[row, idx[row, i], :] = src[row, i, :] (scatter), 16-byte vectors;
// slots outside [0, M) are skipped.
template <bool GATHER>
__global__ __launch_bounds__(256) void kv_copy(uint4* __restrict__ cache,
                                               const int32_t* __restrict__ idx,
                                               uint4* __restrict__ rows, int M, int k, int vecs) {
  const size_t row = blockIdx.y;
  const size_t n = (size_t)k * vecs;
  for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (size_t)gridDim.x * blockDim.x) {
    const int i = (int)(e / vecs), c = (int)(e % vecs);
    const int slot = idx[row * k + i];
    if ((unsigned)slot >= (unsigned)M) continue;
    uint4* cell = cache + (row * M + slot) * vecs + c;
    uint4* r = rows + (row * k + i) * vecs + c;
    if (GATHER) *r = *cell;
    else *cell = *r;
  }
}

}  // namespace

hipError_t launch_sdpa_backward(const Shape& s, int dtype, const void* q, const void* kc,
                                const void* vc, const void* kn, const void* vn, KeyPos kp,
                                const float* lse, const void* dout, void* dq, void* dkc,
                                void* dvc, void* dkn, void* dvn, float* dot, float scale,
                                hipStream_t st) {
  if (dtype == 0)
    return s.d == 64 ? run<float, 64>(s, q, kc, vc, kn, vn, kp, lse, dout, dq, dkc, dvc, dkn,
                                      dvn, dot, scale, st)
                     : run<float, 128>(s, q, kc, vc, kn, vn, kp, lse, dout, dq, dkc, dvc, dkn,
                                       dvn, dot, scale, st);
  return s.d == 64 ? run<bf16_t, 64>(s, q, kc, vc, kn, vn, kp, lse, dout, dq, dkc, dvc, dkn,
                                     dvn, dot, scale, st)
                   : run<bf16_t, 128>(s, q, kc, vc, kn, vn, kp, lse, dout, dq, dkc, dvc, dkn,
                                      dvn, dot, scale, st);
}

hipError_t launch_kv_copy(bool gather, void* cache, const int32_t* idx, void* rows, int nrows,
                          int M, int k, int vecs, hipStream_t st) {
  const size_t n = (size_t)k * vecs;
  if (nrows == 0 || n == 0) return hipSuccess;
  size_t bx = (n + 255) / 256;
  if (bx > 1024) bx = 1024;
  const dim3 grid((unsigned)bx, nrows);
  if (gather)
    return launch_kernel(K_KV_COPY, kv_copy<true>, grid, dim3(256), st, (uint4*)cache, idx,
                         (uint4*)rows, M, k, vecs);
  return launch_kernel(K_KV_COPY, kv_copy<false>, grid, dim3(256), st, (uint4*)cache, idx,
                       (uint4*)rows, M, k, vecs);
}

}  // namespace h2o
