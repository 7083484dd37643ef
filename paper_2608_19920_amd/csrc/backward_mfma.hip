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
// Keys pass: a wave owns 16 keys (H2O_BWD_NKB blocks of 16; 16 keep the
// wave at 200 registers, two waves per SIMD) and the waves share 32-row
// Q/dO tiles. Its S and dP are computed in the key-per-lane orientation, so
// P and dS leave the accumulators already laid out as the B operands of the
// dV and dK products (two 16-row blocks per operand), and the transposed dO
// and Q operands again come from transposing LDS reads.
// When the rows passes would have too few blocks to fill the CUs they split
// the key range: D partials are summed in split order (the dq pass's first
// split leaves the sum for the keys pass), dq partials are float32 and
// bwd_dq_reduce adds them in split order.
//
// Masking: key j is visible to chunk position i iff rel_j <= i, with rel_j =
// -1 for a cache slot (chunk mode), j - M for a chunk key, and the slot's
// token position minus pos0 in cache mode. A row that sees nothing has
// lse = -inf and gets P = 0 (its lambda is taken as +inf).
#include <algorithm>

#include "internal.h"
#include "mfma_ops.h"

namespace h2o {
namespace {

using namespace mfma;

constexpr int kW = 4;          // waves per block
constexpr int kNT = 64 * kW;   // threads per block
constexpr int kTile = 32;      // keys (rows passes) or packed rows (keys pass) per LDS tile
constexpr int kPad = 16;       // bf16 past d per LDS row (pitch 288 B at d = 128)
constexpr int kRB = kW * 32;   // packed rows per block of the rows passes (32 per wave)
#ifndef H2O_BWD_NKB   // key blocks of 16 per wave in the keys pass
#define H2O_BWD_NKB 1
#endif

template <int D>
__host__ __device__ constexpr int pitch() { return D + kPad; }

struct BArgs {
  const bf16_t *q, *dout, *kc, *vc, *kn, *vn;
  const float* lse;
  float* dot;    // D partials [ns_dot][BH][R]; D_r sums them in split order
  float* dfin;   // D_r [BH][R]: plane 0 of dot (one split) or a plane after the partials
  float* part;   // dq partials [ns][BH][R][d] when the dq pass is split
  bf16_t *dq, *dkc, *dvc, *dkn, *dvn;
  const int32_t* tp;   // cache mode: token positions [BH][M]; chunk mode nullptr
  int32_t pos0;
  int Hq, Hkv, G, T, M, R, Nk, BH;
  int ns_dot;    // key-range splits of the D pass
  int ns;        // key-range splits of the rows pass being launched
  float c;       // scale * log2(e)
  float scale;
};

// D_r of packed row r of head bh: the split partials added in split order.
__device__ __forceinline__ float row_dot(const BArgs& a, size_t bh, int r) {
  float v = a.dot[bh * a.R + r];
  for (int s = 1; s < a.ns_dot; ++s) v += a.dot[((size_t)s * a.BH + bh) * a.R + r];
  return v;
}

// Element offset / D of packed row r of KV head (b, h) in [B, Hq, T, .].
__device__ __forceinline__ size_t row_off(const BArgs& a, int b, int h, int r) {
  return (size_t)(b * a.Hq + h * a.G + r % a.G) * a.T + r / a.G;
}

// Key j of head bh in [cache || chunk]. The two bases are passed as values
// (not read through BArgs here) so that the choice stays a register select.
template <int D>
__device__ __forceinline__ const bf16_t* key_ptr(const bf16_t* cache, const bf16_t* fresh, int M,
                                                 int T, size_t bh, int j) {
  return j < M ? cache + (bh * M + j) * (size_t)D : fresh + (bh * T + (j - M)) * (size_t)D;
}

// Earliest chunk position that sees key j (T: none), from the slot's token
// position tpj (read only in cache mode, for j < M).
__device__ __forceinline__ int key_rel_of(const BArgs& a, int j, int32_t tpj) {
  if (j >= a.Nk) return a.T;
  if (j >= a.M) return j - a.M;
  if (!a.tp) return -1;
  const long long r = (long long)tpj - a.pos0;
  return r < -1 ? -1 : (r > a.T ? a.T : (int)r);
}
__device__ __forceinline__ int32_t key_tp(const BArgs& a, size_t bh, int j) {
  return (a.tp && j < a.M) ? a.tp[bh * a.M + j] : 0;
}
__device__ __forceinline__ int key_rel(const BArgs& a, size_t bh, int j) {
  return key_rel_of(a, j, key_tp(a, bh, j));
}

// lambda (log2 domain) of a row from its lse; +inf for a row that sees
// nothing or does not exist (lse -inf), so that every P of it is 0.
__device__ __forceinline__ float lambda_of(float lse) {
  return lse > -INFINITY ? lse * kLog2e : INFINITY;
}
__device__ __forceinline__ float row_lambda(const BArgs& a, bool ok, size_t off) {
  return lambda_of(ok ? a.lse[off] : -INFINITY);
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

// 16-byte chunk e of a 32-row tile for this thread of NT: row (tid + e*NT) /
// (D/8), part (tid + e*NT) % (D/8).
template <int D, int NT = kNT>
constexpr int tile_chunks() { return kTile * (D / 8) / NT; }

// Keys [j0, j0 + 32) of head bh into registers (zero past the keys); in
// cache mode threads 0..31 also fetch the keys' token positions (turned into
// rel only when stored, so that no wait for the loads happens here). The
// four bases come in as values so that the cache/chunk choice stays a
// register select.
template <int D, bool CACHE, int NT = kNT>
__device__ __forceinline__ void load_key_tile(u32x4 (&kr)[(tile_chunks<D, NT>())],
                                              u32x4 (&vr)[(tile_chunks<D, NT>())], int& relr,
                                              const bf16_t* kc, const bf16_t* kn,
                                              const bf16_t* vc, const bf16_t* vn, const BArgs& a,
                                              size_t bh, int j0) {
  constexpr int CH = D / 8;
  const int tid = threadIdx.x;
#pragma unroll
  for (int e = 0; e < tile_chunks<D, NT>(); ++e) {
    const int c = tid + e * NT, j = j0 + c / CH, part = c % CH;
    const bool ok = j < a.Nk;
    const int jj = ok ? j : 0;
    kr[e] = load16(key_ptr<D>(kc, kn, a.M, a.T, bh, jj) + part * 8, ok);
    vr[e] = load16(key_ptr<D>(vc, vn, a.M, a.T, bh, jj) + part * 8, ok);
  }
  if (CACHE && tid < kTile) relr = key_tp(a, bh, j0 + tid);
}

// Packed rows [r0, r0 + 32) of head (b, h): q and dout into registers, and in
// threads 0..31 the row's lse (raw, converted when stored), D and chunk
// position.
template <int D, int NT = kNT>
__device__ __forceinline__ void load_row_tile(u32x4 (&qr)[(tile_chunks<D, NT>())],
                                              u32x4 (&orr)[(tile_chunks<D, NT>())], float& lamr,
                                              float& dotr, int& iposr, const BArgs& a, int b,
                                              int h, size_t bh, int r0) {
  constexpr int CH = D / 8;
  const int tid = threadIdx.x;
#pragma unroll
  for (int e = 0; e < tile_chunks<D, NT>(); ++e) {
    const int c = tid + e * NT, r = r0 + c / CH, part = c % CH;
    const bool ok = r < a.R;
    const size_t off = (ok ? row_off(a, b, h, r) : 0) * D + part * 8;
    qr[e] = load16(a.q + off, ok);
    orr[e] = load16(a.dout + off, ok);
  }
  if (tid < kTile) {
    const int r = r0 + tid;
    const bool ok = r < a.R;
    lamr = ok ? a.lse[row_off(a, b, h, r)] : -INFINITY;
    dotr = ok ? a.dfin[bh * a.R + r] : 0.f;
    iposr = ok ? r / a.G : a.T;
  }
}

// Registers of a 32-row tile into two LDS tiles of pitch D + kPad.
template <int D, int NT = kNT>
__device__ __forceinline__ void store_tile(bf16_t* A, bf16_t* B,
                                           const u32x4 (&ra)[(tile_chunks<D, NT>())],
                                           const u32x4 (&rb)[(tile_chunks<D, NT>())]) {
  constexpr int CH = D / 8, P = pitch<D>();
#pragma unroll
  for (int e = 0; e < tile_chunks<D, NT>(); ++e) {
    const int c = threadIdx.x + e * NT, row = c / CH, part = c % CH;
    *reinterpret_cast<u32x4*>(&A[row * P + part * 8]) = ra[e];
    *reinterpret_cast<u32x4*>(&B[row * P + part * 8]) = rb[e];
  }
}

// ---------------------------------------------------------------- rows passes
// NW waves of 32 rows per block (4, or 8 where the plan finds the pass's
// grid fills whole rounds of the CUs).
template <int D, bool DQ, bool CACHE, int NW = kW>
__global__ __launch_bounds__(NW * 64) void bwd_rows(BArgs a) {
  constexpr int NT = NW * 64, RB = NW * 32;
  constexpr int P = pitch<D>(), KS = D / 32, NL = tile_chunks<D, NT>();
  __shared__ __attribute__((aligned(16))) bf16_t Ks[2][kTile * P];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[2][kTile * P];
  __shared__ __attribute__((aligned(16))) int rel_s[2][kTile];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g4 = lane >> 4, l16 = lane & 15;
  int xb, bhi;
  block_coords(xb, bhi);
  const size_t bh = bhi;
  const int b = bhi / a.Hkv, h = bhi % a.Hkv;
  // x = split * (row tiles) + row tile: the blocks of one key range are
  // consecutive, so they share their K/V tiles in one L2; the row tiles go
  // last to first (later chunk rows see more keys: the longest blocks start
  // first and the shortest fill the last partial round)
  const int nrt = (a.R + RB - 1) / RB;
  const int sp = xb / nrt, rblk = (nrt - 1 - xb % nrt) * RB, wrow0 = rblk + wave * 32;
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
    dr[qb] = 0.f;
    if (DQ && ok) {
      dr[qb] = row_dot(a, bh, r);
      // the first split's blocks leave the summed D for the keys pass
      if (a.ns_dot > 1 && sp == 0 && g4 == 0) a.dfin[bh * a.R + r] = dr[qb];
    }
  }

  const int kv_end =
      CACHE ? a.M : kv_end_for_rows(min(rblk + RB, a.R), a.G, a.T, a.M, a.Nk - a.M);
  // this split's share of the block's key tiles (possibly none)
  const int ntiles_all = (kv_end + kTile - 1) / kTile;
  const int tb = (int)((long long)sp * ntiles_all / a.ns);
  const int te = (int)((long long)(sp + 1) * ntiles_all / a.ns);

  // this thread's 16-byte chunks of a tile: row c / CH, part c % CH
  u32x4 kr[NL], vr[NL];
  int relr = 0;
  f32x4 dqacc[D / 16][2];
#pragma unroll
  for (int db = 0; db < D / 16; ++db)
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) dqacc[db][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float dsum[2] = {0.f, 0.f};

  if (tb < te)
    load_key_tile<D, CACHE, NT>(kr, vr, relr, a.kc, a.kn, a.vc, a.vn, a, bh, tb * kTile);
  for (int t = tb; t < te; ++t) {
    const int buf = (t - tb) & 1, j0 = t * kTile;
    store_tile<D, NT>(Ks[buf], Vs[buf], kr, vr);
    if (CACHE && tid < kTile) rel_s[buf][tid] = key_rel_of(a, j0 + tid, relr);
    __syncthreads();
    if (t + 1 < te)
      load_key_tile<D, CACHE, NT>(kr, vr, relr, a.kc, a.kn, a.vc, a.vn, a, bh,
                                  (t + 1) * kTile);
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
      if (a.ns > 1) {   // unscaled float32 partial of this split
        float* dst = a.part + (((size_t)sp * a.BH + bh) * a.R + r) * D + 4 * g4;
#pragma unroll
        for (int db = 0; db < D / 16; ++db)
          *reinterpret_cast<f32x4*>(dst + 16 * db) = dqacc[db][qb];
      } else {
        bf16_t* dst = a.dq + row_off(a, b, h, r) * D + 4 * g4;
#pragma unroll
        for (int db = 0; db < D / 16; ++db) store4(dst + 16 * db, dqacc[db][qb], a.scale);
      }
    } else {
      float v = dsum[qb];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (g4 == 0 && r < a.R) a.dot[((size_t)sp * a.BH + bh) * a.R + r] = v;
    }
  }
}

// ------------------------------------------------------------------ keys pass
// A wave owns NKB*16 keys (NKB key blocks of 16).
template <int D, int NKB, bool CACHE, int NW = kW>
__global__ __launch_bounds__(NW * 64) void bwd_keys(BArgs a) {
  constexpr int NT = NW * 64;
  constexpr int P = pitch<D>(), KS = D / 32, NL = tile_chunks<D, NT>();
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
  const int kblk = xb * (NW * 16 * NKB), kw0 = kblk + wave * 16 * NKB;
  const bool live = kw0 < a.Nk;

  // this lane's keys kw0 + 16kb + l16: K and V as B operands (k = features)
  bf16x8 kf[NKB][KS], vf[NKB][KS];
  int rel[NKB];
#pragma unroll
  for (int kb = 0; kb < NKB; ++kb) {
    const int j = kw0 + 16 * kb + l16;
    const bool ok = j < a.Nk;
    const int jj = ok ? j : 0;
    const bf16_t* kp = key_ptr<D>(a.kc, a.kn, a.M, a.T, bh, jj) + 8 * g4;
    const bf16_t* vp = key_ptr<D>(a.vc, a.vn, a.M, a.T, bh, jj) + 8 * g4;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      kf[kb][s] = __builtin_bit_cast(bf16x8, load16(kp + 32 * s, ok));
      vf[kb][s] = __builtin_bit_cast(bf16x8, load16(vp + 32 * s, ok));
    }
    rel[kb] = key_rel(a, bh, j);
  }
  // the wave's latest key (wave-uniform): row tiles from that position on
  // need no mask
  int relmax = rel[0];
#pragma unroll
  for (int kb = 1; kb < NKB; ++kb) relmax = max(relmax, rel[kb]);
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

  f32x4 dkacc[D / 16][NKB], dvacc[D / 16][NKB];
#pragma unroll
  for (int db = 0; db < D / 16; ++db)
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) dkacc[db][kb] = dvacc[db][kb] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (t0 < t1) load_row_tile<D, NT>(qr, orr, lamr, dotr, iposr, a, b, h, bh, t0 * kTile);
  for (int t = t0; t < t1; ++t) {
    const int buf = (t - t0) & 1;
    store_tile<D, NT>(Qs[buf], Os[buf], qr, orr);
    if (tid < kTile) {
      lam_s[buf][tid] = lambda_of(lamr);
      dot_s[buf][tid] = dotr;
      ipos_s[buf][tid] = iposr;
    }
    __syncthreads();
    if (t + 1 < t1)
      load_row_tile<D, NT>(qr, orr, lamr, dotr, iposr, a, b, h, bh, (t + 1) * kTile);
    if (!live) continue;
    const bf16_t* Qt = Qs[buf];
    const bf16_t* Ot = Os[buf];
    f32x4 sacc[2][NKB], pacc[2][NKB];   // [rb][kb]: rows 16rb + 4g4 + u, key 16kb + l16
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) sacc[rb][kb] = pacc[rb][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        const bf16x8 aq = row_operand(Qt, P, 16 * rb + l16, 32 * s, lane);
        const bf16x8 ad = row_operand(Ot, P, 16 * rb + l16, 32 * s, lane);
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
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
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          float p = __builtin_amdgcn_exp2f(fmaf(sacc[rb][kb][u], a.c, -lam4[u]));
          if (!full && rel[kb] > ip4[u]) p = 0.f;
          pacc[rb][kb][u] = p * (pacc[rb][kb][u] - dot4[u]);
          sacc[rb][kb][u] = p;
        }
    }
    bf16x8 pop[NKB], dsop[NKB];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
      pop[kb] = pack_pair(sacc[0][kb], sacc[1][kb]);
      dsop[kb] = pack_pair(pacc[0][kb], pacc[1][kb]);
    }
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      const bf16x8 ao = tr_operand(Ot, P, db, lane);
      const bf16x8 aq = tr_operand(Qt, P, db, lane);
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        dvacc[db][kb] = mma(ao, pop[kb], dvacc[db][kb]);
        dkacc[db][kb] = mma(aq, dsop[kb], dkacc[db][kb]);
      }
    }
  }

#pragma unroll
  for (int kb = 0; kb < NKB; ++kb) {
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

// dq = scale * (sum of the split partials in split order), as bf16.
template <int D>
__global__ __launch_bounds__(256) void bwd_dq_reduce(BArgs a) {
  const size_t n4 = (size_t)a.BH * a.R * (D / 4), plane = (size_t)a.BH * a.R * D;
  for (size_t e = (size_t)blockIdx.x * 256 + threadIdx.x; e < n4; e += (size_t)gridDim.x * 256) {
    const size_t flat = e * 4, rr = flat / D;
    const int c = (int)(flat % D), r = (int)(rr % a.R), bhi = (int)(rr / a.R);
    f32x4 v = *reinterpret_cast<const f32x4*>(a.part + flat);
    for (int s = 1; s < a.ns; ++s) v += *reinterpret_cast<const f32x4*>(a.part + s * plane + flat);
    store4(a.dq + row_off(a, bhi / a.Hkv, bhi % a.Hkv, r) * D + c, v, a.scale);
  }
}

template <int D, bool CACHE>
hipError_t run(const Shape& s, const BackwardPlan& pl, BArgs a, hipStream_t st) {
  const int BH = s.BH(), nrt = (s.R() + kRB - 1) / kRB;
  a.ns = pl.ns_dot;
  hipError_t e;
  if constexpr (D == 128) {
    if (pl.dot_waves == 8) {
      const int nrt8 = (s.R() + 8 * 32 - 1) / (8 * 32);
      e = launch_kernel(K_BWD_DOT, bwd_rows<D, false, CACHE, 8>, dim3(nrt8 * a.ns, BH),
                        dim3(512), st, a);
    } else {
      e = launch_kernel(K_BWD_DOT, bwd_rows<D, false, CACHE>, dim3(nrt * a.ns, BH), dim3(kNT),
                        st, a);
    }
  } else {
    e = launch_kernel(K_BWD_DOT, bwd_rows<D, false, CACHE>, dim3(nrt * a.ns, BH), dim3(kNT), st,
                      a);
  }
  if (e != hipSuccess) return e;
  a.ns = pl.ns_dq;
  if constexpr (D == 128) {
    if (pl.dq_waves == 8) {
      const int nrt8 = (s.R() + 8 * 32 - 1) / (8 * 32);
      e = launch_kernel(K_BWD_DQ, bwd_rows<D, true, CACHE, 8>, dim3(nrt8 * a.ns, BH), dim3(512),
                        st, a);
    } else {
      e = launch_kernel(K_BWD_DQ, bwd_rows<D, true, CACHE>, dim3(nrt * a.ns, BH), dim3(kNT), st,
                        a);
    }
  } else {
    e = launch_kernel(K_BWD_DQ, bwd_rows<D, true, CACHE>, dim3(nrt * a.ns, BH), dim3(kNT), st, a);
  }
  if (e != hipSuccess) return e;
  if (a.ns > 1) {
    const size_t n4 = (size_t)BH * s.R() * (D / 4);
    const unsigned nb = (unsigned)std::min<size_t>((n4 + 255) / 256, 4096);
    e = launch_kernel(K_BWD_DQ_REDUCE, bwd_dq_reduce<D>, dim3(nb), dim3(256), st, a);
    if (e != hipSuccess) return e;
  }
  if (s.Nk() == 0) return hipSuccess;
  constexpr int NKB = H2O_BWD_NKB;
  const dim3 gkeys((s.Nk() + kW * 16 * NKB - 1) / (kW * 16 * NKB), BH);
  return launch_kernel(K_BWD_DKDV, bwd_keys<D, NKB, CACHE>, gkeys, dim3(kNT), st, a);
}

}  // namespace

#ifndef H2O_DOT8_PER_CU
#define H2O_DOT8_PER_CU 1
#endif
// Splits of the key range of the two rows passes, so that their grids fill
// the CUs (the D pass runs three 4-wave blocks per CU, the dq pass two);
// at least 8 key tiles per split. At d = 128 either pass runs 8-wave blocks
// (one per CU) where those fill whole rounds of the CUs.
BackwardPlan backward_plan(const Shape& s, int dtype) {
  BackwardPlan p{1, 1, 0, 0, 4, 4};
  const size_t BH = s.BH(), R = s.R();
  size_t bytes = align256_size(BH * R * sizeof(float));
  if (dtype == 1 && R > 0) {
    const long long blocks = (long long)((R + kRB - 1) / kRB) * (long long)BH;
    const long long ntiles = (s.Nk() + kTile - 1) / kTile;
    const long long cus = device_cus();
    auto pick = [&](long long nb, long long target) {
      long long ns = (target + nb - 1) / nb;
      ns = std::min(ns, std::max(1LL, ntiles / 8));
      return (int)std::max(1LL, std::min(ns, 8LL));
    };
    p.ns_dot = pick(blocks, 3 * cus);
    p.ns_dq = pick(blocks, 2 * cus);
    // at d = 128 the dq pass runs 8-wave blocks (256 rows, one per CU) where
    // their grid fills whole rounds: the waves sharing a SIMD then come from
    // one block and keep pace at its barriers
    if (s.d == 128) {
      const long long blocks8 = (long long)((R + 8 * 32 - 1) / (8 * 32)) * (long long)BH;
      const int ns8 = pick(blocks8, cus);
      if (blocks8 * ns8 % cus == 0) {
        p.dq_waves = 8;
        p.ns_dq = ns8;
      }
      // the D pass likewise (three waves per SIMD fit, so one 8-wave block per CU)
      const int nsd8 = pick(blocks8, H2O_DOT8_PER_CU * cus);
      if (H2O_DOT8_PER_CU > 0 && blocks8 * nsd8 % (H2O_DOT8_PER_CU * cus) == 0) {
        p.dot_waves = 8;
        p.ns_dot = nsd8;
      }
    }
    // the D partials, and the summed D after them when there are several
    bytes = align256_size((size_t)(p.ns_dot + (p.ns_dot > 1)) * BH * R * sizeof(float));
    if (p.ns_dq > 1) {
      p.off_part = bytes;
      bytes += align256_size((size_t)p.ns_dq * BH * R * s.d * sizeof(float));
    }
  }
  p.bytes = bytes;
  return p;
}

hipError_t launch_sdpa_backward_mfma(const Shape& s, const void* q, const void* kc,
                                     const void* vc, const void* kn, const void* vn, KeyPos kp,
                                     const float* lse, const void* dout, void* dq, void* dkc,
                                     void* dvc, void* dkn, void* dvn, char* ws, float scale,
                                     hipStream_t st) {
  const BackwardPlan pl = backward_plan(s, 1);
  BArgs a;
  a.q = (const bf16_t*)q;
  a.dout = (const bf16_t*)dout;
  a.kc = (const bf16_t*)kc;
  a.vc = (const bf16_t*)vc;
  a.kn = (const bf16_t*)kn;
  a.vn = (const bf16_t*)vn;
  a.lse = lse;
  a.dot = reinterpret_cast<float*>(ws);
  a.dfin = a.dot + (pl.ns_dot > 1 ? (size_t)pl.ns_dot * s.BH() * s.R() : 0);
  a.part = reinterpret_cast<float*>(ws + pl.off_part);
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
  a.BH = s.BH();
  a.ns_dot = pl.ns_dot;
  a.ns = 1;
  a.c = scale * kLog2e;
  a.scale = scale;
  const bool cache = kp.tp != nullptr;
  if (s.d == 64)
    return cache ? run<64, true>(s, pl, a, st) : run<64, false>(s, pl, a, st);
  return cache ? run<128, true>(s, pl, a, st) : run<128, false>(s, pl, a, st);
}

}  // namespace h2o
