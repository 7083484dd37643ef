// Generic SDPA-with-summed-weights kernels (VALU, float32 arithmetic).
//
// Used for float32 inputs (where the result must match float64 to ~1e-6) and
// for bf16 shapes no faster kernel covers. Two passes over the keys of one KV
// head, with the row log-sum-exp computed first (Sec. "FlashAttention for
// Summed Attention Weights": the column sums need the final row normaliser
// lambda_r before exp(A - lambda) can be summed down a column):
//
//   pass A  lse_r = log sum_j exp(s_rj)           (online max/sum)
//   pass B  m_rj = exp(s_rj - lse_r); out_r = sum_j m_rj V_j;
//           per row tile, column partials sum_{r in tile} m_rj
//   reduce  wsum_j = sum over row tiles of the partials
//
// In cache mode the keys are the M cache slots alone, slot j visible to chunk
// position i iff token_pos[j] - pos0 <= i; a row that sees no slot gets
// lse = -inf, out = 0 and adds nothing to the column sums.
//
// Rows of a KV head are packed position-major: r = i*G + g (chunk position i,
// query head hq = h*G + g). One thread owns one packed row; key tiles of
// kTile keys are staged in LDS and shared by the 64 rows of the block.
#include "internal.h"

namespace h2o {
namespace {

constexpr int kRows = 64;   // rows (threads) per block
constexpr int kTile = 32;   // keys per LDS tile

template <typename E>
__device__ __forceinline__ const E* key_ptr(const E* cache, const E* fresh, size_t bh, int j,
                                            int M, int T, int d) {
  return j < M ? cache + (bh * M + j) * (size_t)d : fresh + (bh * T + (j - M)) * (size_t)d;
}

// Stage key/value rows [j0, j0+kTile) of head bh into LDS as float; rows past
// the key count are zero.
template <typename E, int D>
__device__ void stage(float* lds, const E* cache, const E* fresh, size_t bh, int j0, int Nk,
                      int M, int T) {
  for (int e = threadIdx.x; e < kTile * D; e += blockDim.x) {
    int jj = e / D, c = e % D, j = j0 + jj;
    lds[jj * (D + 1) + c] = j < Nk ? load_elem(key_ptr(cache, fresh, bh, j, M, T, D), c) : 0.f;
  }
}

template <typename E, int D>
__global__ __launch_bounds__(kRows) void pass_a(const E* __restrict__ q, const E* __restrict__ kc,
                                                const E* __restrict__ kn, float* __restrict__ lse,
                                                float* __restrict__ lse_ws, int Hq, int Hkv,
                                                int T, int M, int Tk, float scale, KeyPos kp) {
  __shared__ float ks[kTile * (D + 1)];
  const int G = Hq / Hkv, R = G * T, Nk = M + Tk;
  const size_t bh = blockIdx.y;
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  const int r0 = blockIdx.x * kRows, r = r0 + threadIdx.x;
  const bool valid = r < R;
  const int i = valid ? r / G : 0, g = valid ? r % G : 0;
  const size_t qrow = ((size_t)(b * Hq + h * G + g) * T + i) * D;
  float qv[D];
#pragma unroll
  for (int c = 0; c < D; ++c) qv[c] = valid ? load_elem(q, qrow + c) * scale : 0.f;
  const int r1 = min(r0 + kRows, R);
  const int kv_end = kv_end_for_rows(r1, G, T, M, Tk);
  const int32_t* tp = kp.tp ? kp.tp + bh * (size_t)M : nullptr;
  float m = -INFINITY, l = 0.f;
  for (int j0 = 0; j0 < kv_end; j0 += kTile) {
    __syncthreads();
    stage<E, D>(ks, kc, kn, bh, j0, Nk, M, T);
    __syncthreads();
    const int jn = min(kTile, kv_end - j0);
    for (int jj = 0; jj < jn; ++jj) {
      const int j = j0 + jj;
      if (j >= M && j - M > i) break;          // later chunk keys are invisible too
      if (tp && !pos_visible(tp[j], kp.pos0, i)) continue;
      float s = 0.f;
#pragma unroll
      for (int c = 0; c < D; ++c) s = fmaf(qv[c], ks[jj * (D + 1) + c], s);
      if (s > m) {
        l = l * expf(m - s) + 1.f;
        m = s;
      } else {
        l += expf(s - m);
      }
    }
  }
  if (valid) {
    const float v = m + logf(l);
    lse[(size_t)(b * Hq + h * G + g) * T + i] = v;
    lse_ws[bh * R + r] = v;
  }
}

template <typename E, int D>
__global__ __launch_bounds__(kRows) void pass_b(const E* __restrict__ q, const E* __restrict__ kc,
                                                const E* __restrict__ vc, const E* __restrict__ kn,
                                                const E* __restrict__ vn, E* __restrict__ out,
                                                const float* __restrict__ lse_ws,
                                                float* __restrict__ parts, int Hq, int Hkv, int T,
                                                int M, int Tk, float scale, KeyPos kp) {
  __shared__ float ks[kTile * (D + 1)];
  __shared__ float vs[kTile * (D + 1)];
  __shared__ float ps[kRows * (kTile + 1)];
  const int G = Hq / Hkv, R = G * T, Nk = M + Tk;
  const size_t bh = blockIdx.y;
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  const int r0 = blockIdx.x * kRows, r = r0 + threadIdx.x;
  const bool valid = r < R;
  const int i = valid ? r / G : 0, g = valid ? r % G : 0;
  const size_t qrow = ((size_t)(b * Hq + h * G + g) * T + i) * D;
  float qv[D], o[D];
#pragma unroll
  for (int c = 0; c < D; ++c) {
    qv[c] = valid ? load_elem(q, qrow + c) * scale : 0.f;
    o[c] = 0.f;
  }
  const float lam = valid ? lse_ws[bh * R + r] : 0.f;
  const bool live = valid && lam > -INFINITY;   // the row sees at least one key
  const int r1 = min(r0 + kRows, R);
  const int kv_end = kv_end_for_rows(r1, G, T, M, Tk);
  const int32_t* tp = kp.tp ? kp.tp + bh * (size_t)M : nullptr;
  float* prow = parts + ((size_t)blockIdx.x * gridDim.y + bh) * Nk;
  for (int j0 = 0; j0 < kv_end; j0 += kTile) {
    __syncthreads();
    stage<E, D>(ks, kc, kn, bh, j0, Nk, M, T);
    stage<E, D>(vs, vc, vn, bh, j0, Nk, M, T);
    __syncthreads();
    const int jn = min(kTile, kv_end - j0);
    for (int jj = 0; jj < kTile; ++jj) {
      const int j = j0 + jj;
      float p = 0.f;
      if (live && jj < jn && (j < M ? !tp || pos_visible(tp[j], kp.pos0, i) : j - M <= i)) {
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < D; ++c) s = fmaf(qv[c], ks[jj * (D + 1) + c], s);
        p = expf(s - lam);
#pragma unroll
        for (int c = 0; c < D; ++c) o[c] = fmaf(p, vs[jj * (D + 1) + c], o[c]);
      }
      ps[threadIdx.x * (kTile + 1) + jj] = p;
    }
    __syncthreads();
    // column partial: thread t sums key column t over the block's rows
    if (threadIdx.x < jn) {
      float s = 0.f;
      for (int rr = 0; rr < kRows; ++rr) s += ps[rr * (kTile + 1) + threadIdx.x];
      prow[j0 + threadIdx.x] = s;
    }
  }
  if (valid) {
#pragma unroll
    for (int c = 0; c < D; ++c) store_elem(out, qrow + c, o[c]);
  }
}

template <typename E, int D>
hipError_t run(const Shape& s, const Plan& p, const void* q, const void* kc, const void* vc,
               const void* kn, const void* vn, void* out, float* lse, float* wsum, char* ws,
               float scale, KeyPos kp, hipStream_t st, ScoreAcc acc) {
  dim3 grid((s.R() + kRows - 1) / kRows, s.BH());
  float* lse_ws = reinterpret_cast<float*>(ws + p.off_stats);
  float* parts = reinterpret_cast<float*>(ws + p.off_parts);
  hipError_t e = launch_kernel(K_GENERIC_LSE, pass_a<E, D>, grid, dim3(kRows), st, (const E*)q,
                               (const E*)kc, (const E*)kn, lse, lse_ws, s.Hq, s.Hkv, s.T, s.M,
                               s.Tk(), scale, kp);
  if (e != hipSuccess) return e;
  e = launch_kernel(K_GENERIC_MAIN, pass_b<E, D>, grid, dim3(kRows), st, (const E*)q,
                    (const E*)kc, (const E*)vc, (const E*)kn, (const E*)vn, (E*)out,
                    (const float*)lse_ws, parts, s.Hq, s.Hkv, s.T, s.M, s.Tk(), scale, kp);
  if (e != hipSuccess) return e;
  return launch_colsum_reduce(s, p, parts, wsum, st, acc);
}

}  // namespace

hipError_t launch_sdpa_generic(const Shape& s, const Plan& p, int dtype, const void* q,
                               const void* kc, const void* vc, const void* kn, const void* vn,
                               void* out, float* lse, float* wsum, char* ws, float scale,
                               KeyPos kp, hipStream_t st, ScoreAcc acc) {
  auto go = [&](auto run_fn) {
    return run_fn(s, p, q, kc, vc, kn, vn, out, lse, wsum, ws, scale, kp, st, acc);
  };
  if (dtype == 0) return s.d == 64 ? go(run<float, 64>) : go(run<float, 128>);
  return s.d == 64 ? go(run<bf16_t, 64>) : go(run<bf16_t, 128>);
}

}  // namespace h2o
