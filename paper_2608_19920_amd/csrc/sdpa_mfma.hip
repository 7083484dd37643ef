// bf16 MFMA kernels for the chunk SDPA with summed attention weights (gfx950).
//
// The column sums sum_i m_{i,j} need each row's final normaliser lambda_i
// before exp(A - lambda) can be added down a column (Sec. "FlashAttention for
// Summed Attention Weights"). Here lambda is computed first and the rest in a
// second sweep that has exact probabilities:
//
//   pass A   per packed row r: (m_r, l_r) with lambda_r = m_r + log2 l_r
//            (log2 domain), over this block's key range (one partial per split)
//   pass B   P = exp2(S*c - lambda) on the same S; O += P V; per-wave column
//            partials of P; O written directly (one split) or as a float32
//            partial per split
//   finish   column partials -> wsum (fixed order); split partials of O -> out
//
// Matrix products use v_mfma_f32_16x16x32_bf16 in the S^T = K Q^T
// orientation. For a 16(key) x 16(query) block the accumulator lane l holds
// keys 4*(l/16)+r (r = 0..3) of query l%16, which is exactly the layout of a
// B operand of the next product O^T = V^T P^T (32 keys per MFMA), so P never
// leaves registers. V^T is staged in LDS with the keys of each 32-key tile
// permuted to match that layout. Row statistics reduce inside a lane; the
// column sums reduce across the 16 lanes of a DPP row.
//
// Workgroup: NW waves, each owning NQB*16 consecutive packed rows
// (r = i*G + g: chunk position i, query head h*G+g); all waves share one
// 32-key K/V tile in LDS, so the K/V of a KV head is staged once for the G
// query heads of its group.
#include "internal.h"

namespace h2o {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));   // 16 bytes, register type

constexpr int BN = 32;   // keys per tile

__device__ __forceinline__ f32x4 mfma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, true));
}
constexpr int kRowMirror = 0x140;
constexpr int kRowHalfMirror = 0x141;
constexpr int kQuadXor1 = 0xB1;   // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;   // quad_perm [2,3,0,1]

// Sum of a[r] (key 4*(l/16)+r, this lane's query) over the 16 lanes of the
// DPP row. Returns, in every lane, the total for key 4*(l/16) + (l%16)/4.
__device__ __forceinline__ float colsum16(float a0, float a1, float a2, float a3, int lane) {
  const bool b3 = lane & 8, b2 = lane & 4;
  const float t0 = b3 ? a2 : a0, t1 = b3 ? a3 : a1;   // kept pair
  const float u0 = b3 ? a0 : a2, u1 = b3 ? a1 : a3;   // pair handed to lane 15-l
  const float x0 = t0 + dpp<kRowMirror>(u0);
  const float x1 = t1 + dpp<kRowMirror>(u1);
  const float keep = b2 ? x1 : x0, send = b2 ? x0 : x1;
  float y = keep + dpp<kRowHalfMirror>(send);
  y += dpp<kQuadXor1>(y);
  y += dpp<kQuadXor2>(y);
  return y;
}

__host__ __device__ constexpr int kstride(int D) { return D + 8; }   // bf16 per K row in LDS


// V operand of O^T = V^T P^T. The V tile sits in LDS like the K tile
// ([key][d]) and the transposing LDS read ds_read_b64_tr_b16 builds the
// operand: within each 16-lane group, lane i receives element
// i%4 of the 8-byte chunks addressed by lanes 4k + i/4, k = 0..3. Lane
// 4k + c of group g therefore addresses row (key) 4g + k, columns
// 16*db + 4c..+3, and lane i ends up with V[4g + k][16*db + i] - the keys of
// k-index (g, k) in the P^T operand.
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

__device__ __forceinline__ s16x4 lds_read_tr16(const bf16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_s16x4*)((__attribute__((address_space(3))) bf16_t*)(p)));
}

template <int D>
__device__ __forceinline__ bf16x8 v_operand(const bf16_t* Vs, int db, int lane) {
  const int g = lane >> 4, i = lane & 15;
  const bf16_t* base = Vs + (4 * g + (i >> 2)) * kstride(D) + 16 * db + 4 * (i & 3);
  const s16x4 lo = lds_read_tr16(base);                       // keys 4g + k
  const s16x4 hi = lds_read_tr16(base + 16 * kstride(D));     // keys 16 + 4g + k
  typedef short s16x8 __attribute__((ext_vector_type(8)));
  const s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

struct Geo {
  int G, T, M, R, Nk;
  const bf16_t* q;
  const bf16_t *kc, *vc, *kn, *vn;
};

__device__ __forceinline__ const bf16_t* kv_row(const bf16_t* cache, const bf16_t* fresh,
                                                size_t bh, int j, int M, int T, int D) {
  return j < M ? cache + (bh * M + j) * (size_t)D : fresh + (bh * T + (j - M)) * (size_t)D;
}

// K/V tiles travel global -> registers -> LDS. The loads for tile t+1 are
// issued before tile t is computed and stored to the other LDS buffer after
// it, so one barrier per tile suffices. Key rows past the last column re-read
// that column (always in bounds); they are masked as invisible chunk keys.
// Thread chunk e covers row (tid + e*NT) / (D/8), 16-byte part (tid + e*NT) % (D/8).
template <int D, int NT>
struct Tile {
  static constexpr int CH = D / 8;          // 16-byte chunks per row
  static constexpr int N = BN * CH / NT;    // chunks per thread per tile
};

template <int D, int NT, int N>
__device__ __forceinline__ void load_rows(u32x4 (&r)[N], const bf16_t* cache,
                                          const bf16_t* fresh, const Geo& g, size_t bh, int j0) {
  constexpr int CH = Tile<D, NT>::CH;
#pragma unroll
  for (int e = 0; e < N; ++e) {
    const int c = threadIdx.x + e * NT, kk = c / CH, part = c % CH;
    const int j = min(j0 + kk, g.Nk - 1);
    r[e] = *reinterpret_cast<const u32x4*>(kv_row(cache, fresh, bh, j, g.M, g.T, D) + part * 8);
  }
}

template <int D, int NT, int N>
__device__ __forceinline__ void store_rows(bf16_t* lds, const u32x4 (&r)[N]) {
  constexpr int CH = Tile<D, NT>::CH;
#pragma unroll
  for (int e = 0; e < N; ++e) {
    const int c = threadIdx.x + e * NT, kk = c / CH, part = c % CH;
    *reinterpret_cast<u32x4*>(lds + kk * kstride(D) + part * 8) = r[e];
  }
}

// Query fragments (B operand of S^T = K Q^T) for this wave's rows.
template <int D, int NQB>
__device__ __forceinline__ void load_q(bf16x8 (&qf)[NQB][D / 32], const Geo& g, int b, int h,
                                       int Hq, int wrow0, int lane) {
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const int r = wrow0 + qb * 16 + (lane & 15);
    const bool ok = r < g.R;
    const int i = ok ? r / g.G : 0, gg = ok ? r % g.G : 0;
    const bf16_t* src = g.q + ((size_t)(b * Hq + h * g.G + gg) * g.T + i) * D + 8 * (lane >> 4);
#pragma unroll
    for (int s = 0; s < D / 32; ++s) {
      const u32x4 v = ok ? *reinterpret_cast<const u32x4*>(src + 32 * s) : u32x4{0u, 0u, 0u, 0u};
      qf[qb][s] = __builtin_bit_cast(bf16x8, v);
    }
  }
}

// S^T blocks for the staged tile: sacc[kb][qb], 16 keys x 16 queries each.
template <int D, int NQB>
__device__ __forceinline__ void scores_tile(f32x4 (&sacc)[2][NQB], const bf16_t* Ks,
                                            const bf16x8 (&qf)[NQB][D / 32], int lane) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) sacc[kb][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < D / 32; ++s) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(
          Ks + (kb * 16 + (lane & 15)) * kstride(D) + 32 * s + 8 * (lane >> 4));
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) sacc[kb][qb] = mfma(a, qf[qb][s], sacc[kb][qb]);
    }
  }
}

// Tiles [t0, t1) of a row tile's key range [0, ntiles*BN) for split sp.
__device__ __forceinline__ void split_range(int ntiles, int nsplit, int sp, int& t0, int& t1) {
  const int per = (ntiles + nsplit - 1) / nsplit;
  t0 = min(ntiles, sp * per);
  t1 = min(ntiles, t0 + per);
}

// ------------------------------------------------------------------ pass A
template <int D, int NW, int NQB>
__global__ __launch_bounds__(NW * 64) void lse_pass(Geo g, int Hq, int Hkv, int nsplit,
                                                    float c_log2, float2* __restrict__ stats) {
  constexpr int NT = NW * 64, ROWS = NW * NQB * 16;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[2][BN * kstride(D)];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rt = blockIdx.x / nsplit, sp = blockIdx.x % nsplit;
  const size_t bh = blockIdx.y;
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  const int row0 = rt * ROWS, wrow0 = row0 + wave * NQB * 16;
  const int kv_end = kv_end_for_rows(min(row0 + ROWS, g.R), g.G, g.T, g.M);
  int t0, t1;
  split_range((kv_end + BN - 1) / BN, nsplit, sp, t0, t1);
  const int i_min = min(wrow0, g.R - 1) / g.G;   // smallest chunk position of this wave

  bf16x8 qf[NQB][D / 32];
  load_q<D, NQB>(qf, g, b, h, Hq, wrow0, lane);
  int qi[NQB];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) qi[qb] = (wrow0 + qb * 16 + (lane & 15)) / g.G;

  float m[NQB], l[NQB];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) { m[qb] = -INFINITY; l[qb] = 0.f; }

  u32x4 pk[Tile<D, NT>::N];
  load_rows<D, NT>(pk, g.kc, g.kn, g, bh, t0 * BN);
  store_rows<D, NT>(Ks[0], pk);
  __syncthreads();
  for (int t = t0; t < t1; ++t) {
    const int j0 = t * BN, cur = (t - t0) & 1;
    load_rows<D, NT>(pk, g.kc, g.kn, g, bh, min(t + 1, t1 - 1) * BN);
    f32x4 sacc[2][NQB];
    scores_tile<D, NQB>(sacc, Ks[cur], qf, lane);
    const bool full = j0 + BN - 1 - g.M <= i_min;
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
      float x[8];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float v = sacc[kb][qb][r] * c_log2;
          if (!full) {
            const int j = j0 + kb * 16 + 4 * (lane >> 4) + r;
            if (j >= g.M && j - g.M > qi[qb]) v = -INFINITY;
          }
          x[kb * 4 + r] = v;
        }
      float tmax = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])),
                         fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
      const float mn = fmaxf(m[qb], tmax);
      const float ms = mn == -INFINITY ? 0.f : mn;
      float acc = l[qb] * __builtin_amdgcn_exp2f(m[qb] - ms);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc += __builtin_amdgcn_exp2f(x[e] - ms);
      l[qb] = acc;
      m[qb] = mn;
    }
    store_rows<D, NT>(Ks[cur ^ 1], pk);
    __syncthreads();
  }
  // merge the four lane groups (disjoint key subsets of the same query)
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      const float m2 = __shfl_xor(m[qb], o, 64), l2 = __shfl_xor(l[qb], o, 64);
      const float mn = fmaxf(m[qb], m2);
      const float ms = mn == -INFINITY ? 0.f : mn;
      l[qb] = l[qb] * __builtin_amdgcn_exp2f(m[qb] - ms) + l2 * __builtin_amdgcn_exp2f(m2 - ms);
      m[qb] = mn;
    }
    const int r = wrow0 + qb * 16 + lane;
    if (lane < 16 && r < g.R) stats[((size_t)sp * gridDim.y + bh) * g.R + r] = make_float2(m[qb], l[qb]);
  }
}

// ------------------------------------------------------------------ pass B
template <int D, int NW, int NQB>
__global__ __launch_bounds__(NW * 64) void main_pass(Geo g, int Hq, int Hkv, int nsplit,
                                                     float c_log2, const float2* __restrict__ stats,
                                                     float* __restrict__ parts,
                                                     bf16_t* __restrict__ out,
                                                     float* __restrict__ opart,
                                                     float* __restrict__ lse_out) {
  constexpr int NT = NW * 64, ROWS = NW * NQB * 16;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[2][BN * kstride(D)];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[2][BN * kstride(D)];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rt = blockIdx.x / nsplit, sp = blockIdx.x % nsplit;
  const size_t bh = blockIdx.y;
  const int BH = gridDim.y;
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  const int row0 = rt * ROWS, wrow0 = row0 + wave * NQB * 16;
  const int kv_end = kv_end_for_rows(min(row0 + ROWS, g.R), g.G, g.T, g.M);
  int t0, t1;
  split_range((kv_end + BN - 1) / BN, nsplit, sp, t0, t1);
  const int i_min = min(wrow0, g.R - 1) / g.G;

  bf16x8 qf[NQB][D / 32];
  load_q<D, NQB>(qf, g, b, h, Hq, wrow0, lane);
  int qi[NQB];
  float lam[NQB];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const int r = wrow0 + qb * 16 + (lane & 15);
    qi[qb] = r / g.G;
    if (r < g.R) {
      float mx = -INFINITY;
      for (int s = 0; s < nsplit; ++s) mx = fmaxf(mx, stats[((size_t)s * BH + bh) * g.R + r].x);
      float L = 0.f;
      for (int s = 0; s < nsplit; ++s) {
        const float2 st = stats[((size_t)s * BH + bh) * g.R + r];
        L += st.y * __builtin_amdgcn_exp2f(st.x - mx);
      }
      lam[qb] = mx + __log2f(L);
    } else {
      lam[qb] = INFINITY;   // padding rows: every probability is 0
    }
    if (sp == 0 && lane < 16 && r < g.R) {
      const int i = r / g.G, gg = r % g.G;
      lse_out[(size_t)(b * Hq + h * g.G + gg) * g.T + i] = lam[qb] * kLn2;
    }
  }

  f32x4 oacc[D / 16][NQB];
#pragma unroll
  for (int db = 0; db < D / 16; ++db)
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) oacc[db][qb] = f32x4{0.f, 0.f, 0.f, 0.f};

  float* prow = parts + ((size_t)(rt * NW + wave) * BH + bh) * g.Nk;

  u32x4 pk[Tile<D, NT>::N], pv[Tile<D, NT>::N];
  load_rows<D, NT>(pk, g.kc, g.kn, g, bh, t0 * BN);
  load_rows<D, NT>(pv, g.vc, g.vn, g, bh, t0 * BN);
  store_rows<D, NT>(Ks[0], pk);
  store_rows<D, NT>(Vs[0], pv);
  __syncthreads();
  for (int t = t0; t < t1; ++t) {
    const int j0 = t * BN, cur = (t - t0) & 1;
    const int jn = min(t + 1, t1 - 1) * BN;
    load_rows<D, NT>(pk, g.kc, g.kn, g, bh, jn);
    load_rows<D, NT>(pv, g.vc, g.vn, g, bh, jn);
    f32x4 sacc[2][NQB];
    scores_tile<D, NQB>(sacc, Ks[cur], qf, lane);
    const bool full = j0 + BN - 1 - g.M <= i_min;
    bf16x8 pb[NQB];
    float cs[2][4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) cs[kb][r] = 0.f;
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float p = __builtin_amdgcn_exp2f(fmaf(sacc[kb][qb][r], c_log2, -lam[qb]));
          if (!full) {
            const int j = j0 + kb * 16 + 4 * (lane >> 4) + r;
            if (j >= g.M && j - g.M > qi[qb]) p = 0.f;
          }
          cs[kb][r] += p;
          pb[qb][kb * 4 + r] = (__bf16)p;
        }
    }
    // column partials over this wave's rows
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const float v = colsum16(cs[kb][0], cs[kb][1], cs[kb][2], cs[kb][3], lane);
      const int j = j0 + kb * 16 + 4 * (lane >> 4) + ((lane & 15) >> 2);
      if ((lane & 3) == 0 && j < g.Nk) prow[j] = v;
    }
    // O^T += V^T P^T
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      const bf16x8 a = v_operand<D>(Vs[cur], db, lane);
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) oacc[db][qb] = mfma(a, pb[qb], oacc[db][qb]);
    }
    store_rows<D, NT>(Ks[cur ^ 1], pk);
    store_rows<D, NT>(Vs[cur ^ 1], pv);
    __syncthreads();
  }
  // write O (lane: query qb*16 + l%16, d = db*16 + 4*(l/16) + r)
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const int r = wrow0 + qb * 16 + (lane & 15);
    if (r >= g.R) continue;
    const int i = r / g.G, gg = r % g.G;
    const size_t orow = ((size_t)(b * Hq + h * g.G + gg) * g.T + i) * D;
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      const int dd = db * 16 + 4 * (lane >> 4);
      if (nsplit == 1) {
        uint2 v;
        v.x = (uint32_t)f32_to_bf16(oacc[db][qb][0]) | ((uint32_t)f32_to_bf16(oacc[db][qb][1]) << 16);
        v.y = (uint32_t)f32_to_bf16(oacc[db][qb][2]) | ((uint32_t)f32_to_bf16(oacc[db][qb][3]) << 16);
        *reinterpret_cast<uint2*>(out + orow + dd) = v;
      } else {
        float* dst = opart + (((size_t)sp * BH + bh) * g.R + r) * D + dd;
        *reinterpret_cast<float4*>(dst) =
            make_float4(oacc[db][qb][0], oacc[db][qb][1], oacc[db][qb][2], oacc[db][qb][3]);
      }
    }
  }
}

// Sum of the per-split O partials, rounded to bf16.
template <int D>
__global__ __launch_bounds__(256) void split_reduce(const float* __restrict__ opart,
                                                    bf16_t* __restrict__ out, int Hq, int Hkv,
                                                    int G, int T, int R, int BH, int nsplit) {
  const size_t e4 = (size_t)blockIdx.x * blockDim.x + threadIdx.x;   // group of 4 values
  const size_t n4 = (size_t)BH * R * D / 4;
  if (e4 >= n4) return;
  const size_t e = e4 * 4;
  const size_t bhr = e / D;
  const int dd = (int)(e % D);
  const int r = (int)(bhr % R);
  const size_t bh = bhr / R;
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int sp = 0; sp < nsplit; ++sp) {
    const float4 v = *reinterpret_cast<const float4*>(opart + (size_t)sp * BH * R * D + e);
    s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
  }
  const int i = r / G, gg = r % G;
  uint2 o;
  o.x = (uint32_t)f32_to_bf16(s.x) | ((uint32_t)f32_to_bf16(s.y) << 16);
  o.y = (uint32_t)f32_to_bf16(s.z) | ((uint32_t)f32_to_bf16(s.w) << 16);
  *reinterpret_cast<uint2*>(out + ((size_t)(b * Hq + h * G + gg) * T + i) * D + dd) = o;
}

template <int D, int NW, int NQB>
hipError_t run(const Shape& s, const Plan& p, const void* q, const void* kc, const void* vc,
               const void* kn, const void* vn, void* out, float* lse, float* wsum, char* ws,
               float scale, hipStream_t st) {
  constexpr int ROWS = NW * NQB * 16;
  Geo g{s.G(), s.T, s.M, s.R(), s.Nk(), (const bf16_t*)q, (const bf16_t*)kc,
        (const bf16_t*)vc, (const bf16_t*)kn, (const bf16_t*)vn};
  const int nrt = (s.R() + ROWS - 1) / ROWS;
  dim3 grid(nrt * p.nsplit, s.BH());
  const float c = scale * kLog2e;
  float2* stats = reinterpret_cast<float2*>(ws + p.off_stats);
  float* parts = reinterpret_cast<float*>(ws + p.off_parts);
  float* opart = reinterpret_cast<float*>(ws + p.off_opart);
  {
    LaunchTimer lt(K_MFMA_LSE, st);
    lse_pass<D, NW, NQB><<<grid, NW * 64, 0, st>>>(g, s.Hq, s.Hkv, p.nsplit, c, stats);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  {
    LaunchTimer lt(K_MFMA_MAIN, st);
    main_pass<D, NW, NQB><<<grid, NW * 64, 0, st>>>(g, s.Hq, s.Hkv, p.nsplit, c, stats, parts,
                                                    (bf16_t*)out, opart, lse);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (p.nsplit > 1) {
    const size_t n4 = (size_t)s.BH() * s.R() * s.d / 4;
    LaunchTimer lt(K_SPLIT_REDUCE, st);
    split_reduce<D><<<(unsigned)((n4 + 255) / 256), 256, 0, st>>>(
        opart, (bf16_t*)out, s.Hq, s.Hkv, s.G(), s.T, s.R(), s.BH(), p.nsplit);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return launch_colsum_reduce(s, p, parts, wsum, st);
}

}  // namespace

// Rows of packed queries per workgroup of the MFMA kernels, and per colsum
// partial (one partial per wave).
int mfma_rows_per_block() { return 2 * 4 * 16; }
int mfma_rows_per_part() { return 4 * 16; }

hipError_t launch_sdpa_mfma(const Shape& s, const Plan& p, const void* q, const void* kc,
                            const void* vc, const void* kn, const void* vn, void* out, float* lse,
                            float* wsum, char* ws, float scale, hipStream_t st) {
  if (s.d == 64) return run<64, 2, 4>(s, p, q, kc, vc, kn, vn, out, lse, wsum, ws, scale, st);
  return run<128, 2, 4>(s, p, q, kc, vc, kn, vn, out, lse, wsum, ws, scale, st);
}

}  // namespace h2o
