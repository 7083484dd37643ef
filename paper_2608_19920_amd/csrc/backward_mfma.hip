// bf16 MFMA kernels for the backward of the chunk attention (gfx950): the
// gradients of backward.hip (Sec. "Fine-Tuning for Sparse Attention"; with
// P = softmax(A), dP = dO V^T, D_r = sum_j P_rj dP_rj and dS = P (dP - D)),
// on v_mfma_f32_16x16x32_bf16 with float32 accumulation.
//
//   rows, pass 1  per packed row: D_r from S^T = K Q^T and dP^T = V dO^T over
//                 the keys the row sees (P and dP in float32, never rounded)
//   rows, pass 2  dQ^T += K^T dS^T, dS formed in float32 with the row's D
//                 and rounded to bf16 once, as the operand of the product
//   keys          per key: S = Q K^T and dP = dO V^T with the key's K and V
//                 held in registers, then dV^T += dO^T P and dK^T += Q^T dS
//
// Rows passes: a wave owns 32 packed rows (their Q and dO are B operands in
// registers); the block's four waves share 32-key K/V tiles in LDS; the
// transposed K operand of the dQ product comes from ds_read_b64_tr_b16.
// Keys pass: a wave owns 32 keys and the waves share 32-row Q/dO tiles. Its
// S and dP are computed in the key-per-lane orientation, so P and dS leave
// the accumulators already laid out as the B operands of the dV and dK
// products (two 16-row blocks per operand), and the transposed dO and Q
// operands again come from transposing LDS reads.
//
// Masking: key j is visible to chunk position i iff rel_j <= i, with rel_j =
// -1 for a cache slot (chunk mode), j - M for a chunk key, and the slot's
// token position minus pos0 in cache mode. A row that sees nothing has
// lse = -inf and gets P = 0 (its lambda is taken as +inf).
#include "internal.h"
#include "mfma_ops.h"

namespace h2o {
namespace {

using namespace mfma;

constexpr int kW = 4;          // waves per block
constexpr int kNT = 64 * kW;   // threads per block
constexpr int kTile = 32;      // keys (rows passes) or packed rows (keys pass) per LDS tile
constexpr int kPad = 16;       // bf16 past d per LDS row (pitch 288 B at d = 128)

template <int D>
__host__ __device__ constexpr int pitch() { return D + kPad; }

struct BArgs {
  const bf16_t *q, *dout, *kc, *vc, *kn, *vn;
  const float* lse;
  float* dot;   // [BH][R]
  bf16_t *dq, *dkc, *dvc, *dkn, *dvn;
  const int32_t* tp;   // cache mode: token positions [BH][M]; chunk mode nullptr
  int32_t pos0;
  int Hq, Hkv, G, T, M, R, Nk;
  float c;       // scale * log2(e)
  float scale;
};

// Element offset / D of packed row r of KV head (b, h) in [B, Hq, T, .].
__device__ __forceinline__ size_t row_off(const BArgs& a, int b, int h, int r) {
  return (size_t)(b * a.Hq + h * a.G + r % a.G) * a.T + r / a.G;
}

template <int D>
__device__ __forceinline__ const bf16_t* key_ptr(const bf16_t* cache, const bf16_t* fresh,
                                                 const BArgs& a, size_t bh, int j) {
  return j < a.M ? cache + (bh * a.M + j) * (size_t)D
                 : fresh + (bh * a.T + (j - a.M)) * (size_t)D;
}

// Earliest chunk position that sees key j (T: none).
__device__ __forceinline__ int key_rel(const BArgs& a, size_t bh, int j) {
  if (j >= a.Nk) return a.T;
  if (j >= a.M) return j - a.M;
  if (!a.tp) return -1;
  const long long r = (long long)a.tp[bh * a.M + j] - a.pos0;
  return r < -1 ? -1 : (r > a.T ? a.T : (int)r);
}

__device__ __forceinline__ float row_lambda(const BArgs& a, bool ok, size_t off) {
  const float l = ok ? a.lse[off] : -INFINITY;
  return l > -INFINITY ? l * kLog2e : INFINITY;
}

__device__ __forceinline__ u32x4 load16(const bf16_t* p, bool ok) {
  return ok ? *reinterpret_cast<const u32x4*>(p) : u32x4{0u, 0u, 0u, 0u};
}

// Workgroups reach the 8 XCDs round-robin in dispatch order. When the heads
// divide evenly over the XCDs, all blocks of one head are given consecutive
// slots of one XCD, so the tiles they share stay in that XCD's L2.
constexpr int kXcds = 8;
__device__ __forceinline__ void block_coords(int& x, int& bh) {
  const int nx = gridDim.x, lin = blockIdx.x + blockIdx.y * gridDim.x;
  if (gridDim.y % kXcds == 0) {
    const int i = lin / kXcds;
    bh = (i / nx) * kXcds + lin % kXcds;
    x = i % nx;
  } else {
    bh = blockIdx.y;
    x = blockIdx.x;
  }
}

// Store 4 consecutive gradient elements (one lane's C values) as bf16.
__device__ __forceinline__ void store4(bf16_t* p, const f32x4& v, float mul) {
  typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
  u16x4 r;
#pragma unroll
  for (int u = 0; u < 4; ++u) r[u] = __builtin_bit_cast(uint16_t, (__bf16)(v[u] * mul));
  *reinterpret_cast<u16x4*>(p) = r;
}

// ---------------------------------------------------------------- rows passes
template <int D, bool DQ, bool CACHE>
__global__ __launch_bounds__(kNT) void bwd_rows(BArgs a) {
  constexpr int P = pitch<D>(), KS = D / 32, CH = D / 8, NL = kTile * CH / kNT;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[2][kTile * P];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[2][kTile * P];
  __shared__ __attribute__((aligned(16))) int rel_s[2][kTile];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g4 = lane >> 4, l16 = lane & 15;
  int xb, bhi;
  block_coords(xb, bhi);
  const size_t bh = bhi;
  const int b = bhi / a.Hkv, h = bhi % a.Hkv;
  const int rblk = xb * (kW * 32), wrow0 = rblk + wave * 32;
  const bool live = wrow0 < a.R;
  const int imin = wrow0 / a.G;

  bf16x8 qf[2][KS], df[2][KS];
  float lam[2], dr[2];
  int ipos[2];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int r = wrow0 + 16 * qb + l16;
    const bool ok = r < a.R;
    const size_t off = ok ? row_off(a, b, h, r) : 0;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      qf[qb][s] = __builtin_bit_cast(bf16x8, load16(a.q + off * D + 32 * s + 8 * g4, ok));
      df[qb][s] = __builtin_bit_cast(bf16x8, load16(a.dout + off * D + 32 * s + 8 * g4, ok));
    }
    lam[qb] = row_lambda(a, ok, off);
    ipos[qb] = ok ? r / a.G : 0;
    dr[qb] = (DQ && ok) ? a.dot[bh * a.R + r] : 0.f;
  }

  const int kv_end =
      CACHE ? a.M : kv_end_for_rows(min(rblk + kW * 32, a.R), a.G, a.T, a.M, a.Nk - a.M);
  const int ntiles = (kv_end + kTile - 1) / kTile;
  const bf16_t* kc_bh = a.kc;
  const bf16_t* vc_bh = a.vc;

  // this thread's 16-byte chunks of a tile: row c / CH, part c % CH
  u32x4 kr[NL], vr[NL];
  int relr = 0;
  auto load = [&](int t) {
#pragma unroll
    for (int e = 0; e < NL; ++e) {
      const int c = tid + e * kNT, j = t * kTile + c / CH, part = c % CH;
      const bool ok = j < a.Nk;
      const int jj = ok ? j : 0;
      kr[e] = load16(key_ptr<D>(kc_bh, a.kn, a, bh, jj) + part * 8, ok);
      vr[e] = load16(key_ptr<D>(vc_bh, a.vn, a, bh, jj) + part * 8, ok);
    }
    if (CACHE && tid < kTile) relr = key_rel(a, bh, t * kTile + tid);
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int e = 0; e < NL; ++e) {
      const int c = tid + e * kNT, row = c / CH, part = c % CH;
      *reinterpret_cast<u32x4*>(&Ks[buf][row * P + part * 8]) = kr[e];
      *reinterpret_cast<u32x4*>(&Vs[buf][row * P + part * 8]) = vr[e];
    }
    if (CACHE && tid < kTile) rel_s[buf][tid] = relr;
  };

  f32x4 dqacc[D / 16][2];
#pragma unroll
  for (int db = 0; db < D / 16; ++db)
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) dqacc[db][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float dsum[2] = {0.f, 0.f};

  if (ntiles > 0) load(0);
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1, j0 = t * kTile;
    store(buf);
    __syncthreads();
    if (t + 1 < ntiles) load(t + 1);
    if (!live) continue;
    const bf16_t* Kt = Ks[buf];
    const bf16_t* Vt = Vs[buf];
    f32x4 sacc[2][2], pacc[2][2];   // [kb][qb]: keys 16kb + 4g4 + u, query l16
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) sacc[kb][qb] = pacc[kb][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8 ak = row_operand(Kt, P, 16 * kb + l16, 32 * s, lane);
        const bf16x8 av = row_operand(Vt, P, 16 * kb + l16, 32 * s, lane);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
          sacc[kb][qb] = mma(ak, qf[qb][s], sacc[kb][qb]);
          pacc[kb][qb] = mma(av, df[qb][s], pacc[kb][qb]);
        }
      }
    // wave-uniform: every key of the tile visible to every row of the wave
    const bool full = !CACHE && j0 + kTile - 1 - a.M <= imin;
    int rel[2][4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int jl = 16 * kb + 4 * g4 + u, j = j0 + jl;
        rel[kb][u] = CACHE ? rel_s[buf][jl] : (j < a.M ? -1 : j - a.M);
      }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          float p = __builtin_amdgcn_exp2f(fmaf(sacc[kb][qb][u], a.c, -lam[qb]));
          if (!full && rel[kb][u] > ipos[qb]) p = 0.f;
          if (DQ) sacc[kb][qb][u] = p * (pacc[kb][qb][u] - dr[qb]);
          else dsum[qb] = fmaf(p, pacc[kb][qb][u], dsum[qb]);
        }
    if (DQ) {
      bf16x8 dsop[2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) dsop[qb] = pack_pair(sacc[0][qb], sacc[1][qb]);
#pragma unroll
      for (int db = 0; db < D / 16; ++db) {
        const bf16x8 ak = tr_operand(Kt, P, db, lane);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) dqacc[db][qb] = mma(ak, dsop[qb], dqacc[db][qb]);
      }
    }
  }

#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int r = wrow0 + 16 * qb + l16;
    if (DQ) {
      if (r >= a.R) continue;
      bf16_t* dst = a.dq + row_off(a, b, h, r) * D + 4 * g4;
#pragma unroll
      for (int db = 0; db < D / 16; ++db) store4(dst + 16 * db, dqacc[db][qb], a.scale);
    } else {
      float v = dsum[qb];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (g4 == 0 && r < a.R) a.dot[bh * a.R + r] = v;
    }
  }
}

// ------------------------------------------------------------------ keys pass
template <int D, bool CACHE>
__global__ __launch_bounds__(kNT) void bwd_keys(BArgs a) {
  constexpr int P = pitch<D>(), KS = D / 32, CH = D / 8, NL = kTile * CH / kNT;
  __shared__ __attribute__((aligned(16))) bf16_t Qs[2][kTile * P];
  __shared__ __attribute__((aligned(16))) bf16_t Os[2][kTile * P];
  __shared__ __attribute__((aligned(16))) float lam_s[2][kTile];
  __shared__ __attribute__((aligned(16))) float dot_s[2][kTile];
  __shared__ __attribute__((aligned(16))) int ipos_s[2][kTile];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g4 = lane >> 4, l16 = lane & 15;
  int xb, bhi;
  block_coords(xb, bhi);
  const size_t bh = bhi;
  const int b = bhi / a.Hkv, h = bhi % a.Hkv;
  const int kblk = xb * (kW * 32), kw0 = kblk + wave * 32;
  const bool live = kw0 < a.Nk;

  // this lane's keys kw0 + 16kb + l16: K and V as B operands (k = features)
  bf16x8 kf[2][KS], vf[2][KS];
  int rel[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int j = kw0 + 16 * kb + l16;
    const bool ok = j < a.Nk;
    const int jj = ok ? j : 0;
    const bf16_t* kp = key_ptr<D>(a.kc, a.kn, a, bh, jj) + 8 * g4;
    const bf16_t* vp = key_ptr<D>(a.vc, a.vn, a, bh, jj) + 8 * g4;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      kf[kb][s] = __builtin_bit_cast(bf16x8, load16(kp + 32 * s, ok));
      vf[kb][s] = __builtin_bit_cast(bf16x8, load16(vp + 32 * s, ok));
    }
    rel[kb] = key_rel(a, bh, j);
  }
  // the wave's latest key (wave-uniform): row tiles from that position on
  // need no mask
  int relmax = max(rel[0], rel[1]);
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) relmax = max(relmax, __shfl_xor(relmax, o));

  // the block's first row tile that may see one of its keys (chunk mode: the
  // first chunk key of the block; cache mode: row 0)
  const int rel_first = CACHE ? -1 : (kblk < a.M ? -1 : kblk - a.M);
  const int t0 = (rel_first < 0 ? 0 : rel_first * a.G) / kTile;
  const int t1 = (a.R + kTile - 1) / kTile;

  u32x4 qr[NL], orr[NL];
  float lamr = 0.f, dotr = 0.f;
  int iposr = 0;
  auto load = [&](int t) {
    const int r0 = t * kTile;
#pragma unroll
    for (int e = 0; e < NL; ++e) {
      const int c = tid + e * kNT, r = r0 + c / CH, part = c % CH;
      const bool ok = r < a.R;
      const size_t off = (ok ? row_off(a, b, h, r) : 0) * D + part * 8;
      qr[e] = load16(a.q + off, ok);
      orr[e] = load16(a.dout + off, ok);
    }
    if (tid < kTile) {
      const int r = r0 + tid;
      const bool ok = r < a.R;
      lamr = row_lambda(a, ok, ok ? row_off(a, b, h, r) : 0);
      dotr = ok ? a.dot[bh * a.R + r] : 0.f;
      iposr = ok ? r / a.G : a.T;
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int e = 0; e < NL; ++e) {
      const int c = tid + e * kNT, row = c / CH, part = c % CH;
      *reinterpret_cast<u32x4*>(&Qs[buf][row * P + part * 8]) = qr[e];
      *reinterpret_cast<u32x4*>(&Os[buf][row * P + part * 8]) = orr[e];
    }
    if (tid < kTile) {
      lam_s[buf][tid] = lamr;
      dot_s[buf][tid] = dotr;
      ipos_s[buf][tid] = iposr;
    }
  };

  f32x4 dkacc[D / 16][2], dvacc[D / 16][2];
#pragma unroll
  for (int db = 0; db < D / 16; ++db)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) dkacc[db][kb] = dvacc[db][kb] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (t0 < t1) load(t0);
  for (int t = t0; t < t1; ++t) {
    const int buf = (t - t0) & 1;
    store(buf);
    __syncthreads();
    if (t + 1 < t1) load(t + 1);
    if (!live) continue;
    const bf16_t* Qt = Qs[buf];
    const bf16_t* Ot = Os[buf];
    f32x4 sacc[2][2], pacc[2][2];   // [rb][kb]: rows 16rb + 4g4 + u, key 16kb + l16
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) sacc[rb][kb] = pacc[rb][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        const bf16x8 aq = row_operand(Qt, P, 16 * rb + l16, 32 * s, lane);
        const bf16x8 ad = row_operand(Ot, P, 16 * rb + l16, 32 * s, lane);
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          sacc[rb][kb] = mma(aq, kf[kb][s], sacc[rb][kb]);
          pacc[rb][kb] = mma(ad, vf[kb][s], pacc[rb][kb]);
        }
      }
    const bool full = relmax <= (t * kTile) / a.G;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const f32x4 lam4 = *reinterpret_cast<const f32x4*>(&lam_s[buf][16 * rb + 4 * g4]);
      const f32x4 dot4 = *reinterpret_cast<const f32x4*>(&dot_s[buf][16 * rb + 4 * g4]);
      int ip4[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) ip4[u] = ipos_s[buf][16 * rb + 4 * g4 + u];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          float p = __builtin_amdgcn_exp2f(fmaf(sacc[rb][kb][u], a.c, -lam4[u]));
          if (!full && rel[kb] > ip4[u]) p = 0.f;
          pacc[rb][kb][u] = p * (pacc[rb][kb][u] - dot4[u]);
          sacc[rb][kb][u] = p;
        }
    }
    bf16x8 pop[2], dsop[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      pop[kb] = pack_pair(sacc[0][kb], sacc[1][kb]);
      dsop[kb] = pack_pair(pacc[0][kb], pacc[1][kb]);
    }
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      const bf16x8 ao = tr_operand(Ot, P, db, lane);
      const bf16x8 aq = tr_operand(Qt, P, db, lane);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        dvacc[db][kb] = mma(ao, pop[kb], dvacc[db][kb]);
        dkacc[db][kb] = mma(aq, dsop[kb], dkacc[db][kb]);
      }
    }
  }

#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int j = kw0 + 16 * kb + l16;
    if (j >= a.Nk) continue;
    bf16_t* dk = j < a.M ? a.dkc + (bh * a.M + j) * (size_t)D
                         : a.dkn + (bh * a.T + (j - a.M)) * (size_t)D;
    bf16_t* dv = j < a.M ? a.dvc + (bh * a.M + j) * (size_t)D
                         : a.dvn + (bh * a.T + (j - a.M)) * (size_t)D;
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      store4(dk + 16 * db + 4 * g4, dkacc[db][kb], a.scale);
      store4(dv + 16 * db + 4 * g4, dvacc[db][kb], 1.f);
    }
  }
}

template <int D, bool CACHE>
hipError_t run(const Shape& s, const BArgs& a, hipStream_t st) {
  const int BH = s.BH();
  const dim3 grows((s.R() + kW * 32 - 1) / (kW * 32), BH);
  hipError_t e = launch_kernel(K_BWD_DOT, bwd_rows<D, false, CACHE>, grows, dim3(kNT), st, a);
  if (e != hipSuccess) return e;
  e = launch_kernel(K_BWD_DQ, bwd_rows<D, true, CACHE>, grows, dim3(kNT), st, a);
  if (e != hipSuccess || s.Nk() == 0) return e;
  const dim3 gkeys((s.Nk() + kW * 32 - 1) / (kW * 32), BH);
  return launch_kernel(K_BWD_DKDV, bwd_keys<D, CACHE>, gkeys, dim3(kNT), st, a);
}

}  // namespace

hipError_t launch_sdpa_backward_mfma(const Shape& s, const void* q, const void* kc,
                                     const void* vc, const void* kn, const void* vn, KeyPos kp,
                                     const float* lse, const void* dout, void* dq, void* dkc,
                                     void* dvc, void* dkn, void* dvn, float* dot, float scale,
                                     hipStream_t st) {
  BArgs a;
  a.q = (const bf16_t*)q;
  a.dout = (const bf16_t*)dout;
  a.kc = (const bf16_t*)kc;
  a.vc = (const bf16_t*)vc;
  a.kn = (const bf16_t*)kn;
  a.vn = (const bf16_t*)vn;
  a.lse = lse;
  a.dot = dot;
  a.dq = (bf16_t*)dq;
  a.dkc = (bf16_t*)dkc;
  a.dvc = (bf16_t*)dvc;
  a.dkn = (bf16_t*)dkn;
  a.dvn = (bf16_t*)dvn;
  a.tp = kp.tp;
  a.pos0 = kp.pos0;
  a.Hq = s.Hq;
  a.Hkv = s.Hkv;
  a.G = s.G();
  a.T = s.T;
  a.M = s.M;
  a.R = s.R();
  a.Nk = s.Nk();
  a.c = scale * kLog2e;
  a.scale = scale;
  const bool cache = kp.tp != nullptr;
  if (s.d == 64)
    return cache ? run<64, true>(s, a, st) : run<64, false>(s, a, st);
  return cache ? run<128, true>(s, a, st) : run<128, false>(s, a, st);
}

}  // namespace h2o
