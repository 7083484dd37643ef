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
// leaves registers. Row statistics reduce inside a lane; the column sums
// reduce across the 16 lanes of a DPP row.
//
// Workgroup: NW waves, each owning NQB*16 consecutive packed rows
// (r = i*G + g: chunk position i, query head h*G+g); all waves share one
// 32-key K/V tile in LDS, so the K/V of a KV head is staged once for the G
// query heads of its group. Tiles are triple buffered in LDS (see the
// software pipeline below).
#include "internal.h"

#include <climits>
#include <type_traits>

namespace h2o {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));   // 16 bytes, register type
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

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
// Each step hands half of the remaining values to the partner lane and keeps
// the other half, so 4 values need 6 + 3 + 2 operations.
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

#ifndef H2O_KPAD
#define H2O_KPAD 16
#endif
#ifndef H2O_VPAD
#define H2O_VPAD 16
#endif
// bf16 per LDS row of the K and V tiles (row pitch 288 bytes at d=128; both
// pitches make the operand reads and the tile stores free of bank conflicts)
__host__ __device__ constexpr int kstride(int D) { return D + H2O_KPAD; }
__host__ __device__ constexpr int vstride(int D) { return D + H2O_VPAD; }

// V operand of O^T = V^T P^T. The V tile sits in LDS like the K tile
// ([key][d]) and the transposing LDS read ds_read_b64_tr_b16 builds the
// operand: within each 16-lane group, lane i receives element i%4 of the
// 8-byte chunks addressed by lanes 4k + i/4, k = 0..3. Lane 4k + c of group
// g therefore addresses row (key) 4g + k, columns 16*db + 4c..+3, and lane i
// ends up with V[4g + k][16*db + i] - the keys of k-index (g, k) in the P^T
// operand; a second read covers keys 16 + 4g + k.
__device__ __forceinline__ s16x4 lds_read_tr16(const bf16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_s16x4*)((__attribute__((address_space(3))) bf16_t*)(p)));
}

template <int D>
__device__ __forceinline__ bf16x8 v_operand(const bf16_t* Vs, int db, int lane) {
  const int g = lane >> 4, i = lane & 15;
  const bf16_t* base = Vs + (4 * g + (i >> 2)) * vstride(D) + 16 * db + 4 * (i & 3);
  const s16x4 lo = lds_read_tr16(base);
  const s16x4 hi = lds_read_tr16(base + 16 * vstride(D));
  const s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

struct Geo {
  int G, T, M, R, Nk, Tk;   // Tk: chunk key columns (T, or 0 in cache mode)
  const bf16_t* q;
  const bf16_t *kc, *vc, *kn, *vn;
  const int32_t* tp;        // cache mode: token positions [BH][M]
  int32_t pos0;
};

// ------------------------------------------------------------ tile staging
// Thread chunk e of a tile is row (tid + e*NT) / (D/8), 16-byte part
// (tid + e*NT) % (D/8); its byte offset inside a tile of global rows and
// inside an LDS tile is fixed per thread, so a tile load is a uniform base
// plus constant offsets. Rows past the last key column re-read that column
// (always in bounds); they are masked as invisible chunk keys.
template <int D, int NT>
struct Tile {
  static constexpr int CH = D / 8;
  static constexpr int N = BN * CH / NT;
  uint32_t goff[N];   // bytes from the tile's first global row
  uint32_t loff[N];   // bytes from the LDS tile base (K tiles)
  uint32_t vloff[N];  // bytes from the LDS tile base (V tiles)
  int row[N], part[N];
  __device__ __forceinline__ Tile() {
#pragma unroll
    for (int e = 0; e < N; ++e) {
      const int c = threadIdx.x + e * NT;
      row[e] = c / CH;
      part[e] = c % CH;
      goff[e] = (uint32_t)(row[e] * D + part[e] * 8) * 2u;
      loff[e] = (uint32_t)(row[e] * kstride(D) + part[e] * 8) * 2u;
      vloff[e] = (uint32_t)(row[e] * vstride(D) + part[e] * 8) * 2u;
    }
  }
};

// PURE: the caller knows the tile is wholly inside the cache or wholly
// inside the chunk, and the load takes no branch.
template <int D, int NT, bool PURE = false, int N>
__device__ __forceinline__ void load_tile(u32x4 (&r)[N], const Tile<D, NT>& tl,
                                          const bf16_t* cache_bh, const bf16_t* fresh_bh, int j0,
                                          int M, int Nk) {
  // Tiles wholly inside the cache or wholly inside the chunk have one base row.
  const bool in_cache = j0 + BN <= M, in_chunk = j0 >= M && j0 + BN <= Nk;
  if (PURE || in_cache || in_chunk) {
    const char* base = reinterpret_cast<const char*>(
        in_cache ? cache_bh + (size_t)j0 * D : fresh_bh + (size_t)(j0 - M) * D);
#pragma unroll
    for (int e = 0; e < N; ++e) r[e] = *reinterpret_cast<const u32x4*>(base + tl.goff[e]);
  } else {
#pragma unroll
    for (int e = 0; e < N; ++e) {
      const int j = min(j0 + tl.row[e], Nk - 1);
      const bf16_t* p = j < M ? cache_bh + (size_t)j * D : fresh_bh + (size_t)(j - M) * D;
      r[e] = *reinterpret_cast<const u32x4*>(p + tl.part[e] * 8);
    }
  }
}

template <int D, int NT, int N>
__device__ __forceinline__ void store_tile(bf16_t* lds, const uint32_t (&off)[N],
                                           const u32x4 (&r)[N]) {
  char* base = reinterpret_cast<char*>(lds);
#pragma unroll
  for (int e = 0; e < N; ++e) *reinterpret_cast<u32x4*>(base + off[e]) = r[e];
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

// Key column j of a chunk is visible to chunk position i iff j < M or j-M <= i.
__device__ __forceinline__ bool visible(int j, int M, int i) { return j < M || j - M <= i; }

// Masking of a tile: MK = 0 none, 1 the chunk's causal rule (visible()), 2
// cache mode, where each key's position relative to the chunk, rp =
// token_pos - pos0 (a value above every chunk position past the cache), is
// staged in LDS with the tile and the key is visible to position i iff
// rp <= i; 3 cache mode on a tile every row of the wave sees (positions
// still staged for the tiles ahead, no mask). Rel holds the rp of this
// lane's 8 keys of the tile.
struct Rel {
  int rp[2][4];
};
constexpr int kRpFar = 1 << 30;   // above every chunk position
// ints per staged row of relative positions: the tile's BN positions, then
// (at index BN) their maximum, which lets a wave whose rows all see every
// key of the tile skip the mask (16-byte aligned rows)
constexpr int kRpPitch = BN + 4;

__device__ __forceinline__ void load_rel(Rel& rl, const int* rps, int lane) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int4 v = *reinterpret_cast<const int4*>(rps + 16 * kb + 4 * (lane >> 4));
    rl.rp[kb][0] = v.x;
    rl.rp[kb][1] = v.y;
    rl.rp[kb][2] = v.z;
    rl.rp[kb][3] = v.w;
  }
}

template <int MK>
__device__ __forceinline__ bool key_hidden(const Rel& rl, int kb, int r, int j, int M, int i) {
  if (MK == 1) return !visible(j, M, i);
  if (MK == 2) return rl.rp[kb][r] > i;
  return false;
}

// Cache mode: thread tid < BN fetches the token position of key j0 + tid.
// It becomes a relative position (kRpFar past the cache) only when the tile
// is stored: arithmetic on the loaded value where the load is issued would
// wait for it, and with it for the K/V loads issued just before.
__device__ __forceinline__ int32_t load_tp(const int32_t* tp_bh, int j0, int M) {
  const int j = j0 + (int)threadIdx.x;
  return (threadIdx.x < BN && j < M) ? tp_bh[j] : 0;
}
template <bool MAX>
__device__ __forceinline__ void store_rp(int* rps, int32_t tpj, int32_t pos0, int j0, int M) {
  // an empty asm that takes and returns the value: the conversion below
  // cannot be moved (or folded into the load) ahead of this point
  asm volatile("" : "+v"(tpj));
  int v = -kRpFar;
  if (threadIdx.x < BN) {
    const int j = j0 + (int)threadIdx.x;
    const long long r = (long long)tpj - pos0;
    v = j >= M ? kRpFar : (r > kRpFar ? kRpFar : (r < -kRpFar ? -kRpFar : (int)r));
    rps[threadIdx.x] = v;
  }
  if (MAX && threadIdx.x < 64) {   // wave 0: the maximum over lanes 0 .. BN-1
#pragma unroll
    for (int o = 1; o < BN; o <<= 1) v = max(v, __shfl_xor(v, o, 64));
    if (threadIdx.x == 0) rps[BN] = v;
  }
}

// Cache mode: whether some row of the wave cannot see some key of the tile
// (its largest relative position exceeds the wave's first chunk position,
// qi[0] of lane 0). Wave-uniform.
template <int NQB>
__device__ __forceinline__ bool tile_needs_mask(const int* rps, const int (&qi)[NQB]) {
  return __builtin_amdgcn_readfirstlane(rps[BN]) > __builtin_amdgcn_readfirstlane(qi[0]);
}

// Tiles [t0, t1) of a row tile's key range [0, ntiles*BN) for split sp.
__device__ __forceinline__ void split_range(int ntiles, int nsplit, int sp, int& t0, int& t1) {
  const int per = (ntiles + nsplit - 1) / nsplit;
  t0 = min(ntiles, sp * per);
  t1 = min(ntiles, t0 + per);
}

// Tiles are software pipelined over three LDS buffers: while the softmax
// arithmetic of tile t runs, the MFMAs of S(t+1) are issued from the buffer
// already holding tile t+1, the rows of tile t+2 (loaded one tile earlier)
// go from registers to the buffer tile t-1 used, and the global loads of
// tile t+3 are issued into a second register set. One barrier per tile
// orders the buffer reuse. Tiles whose columns some row of the block cannot see run
// in a second loop with the causal mask applied; each loop body is straight
// line so the compiler can interleave MFMA and VALU work.
constexpr int NBUF = 3;

// Instruction interleaving hints for the straight-line tile bodies:
// sched_group_barrier(mask, n, id) asks the scheduler for n instructions of a
// class (0x2 VALU, 0x8 MFMA) in order. The MFMAs of S(t+1) do not depend on
// the softmax arithmetic of tile t, so they alternate with it.
#ifndef H2O_INTERLEAVE
#define H2O_INTERLEAVE 0
#endif
template <int NMFMA, int NVALU>
__device__ __forceinline__ void interleave() {
  if (!H2O_INTERLEAVE) return;
#pragma unroll
  for (int i = 0; i < NMFMA; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, NVALU, 0);
  }
}

// First tile index at which some row of the block may see an invisible
// column: tile t needs the mask iff t*BN + BN-1 - M > i_min.
__device__ __forceinline__ int first_masked_tile(int M, int i_min) {
  const int x = M + i_min - (BN - 1);          // mask needed iff t*BN > x
  return x < 0 ? 0 : x / BN + 1;
}

// ------------------------------------------------------------ block order
// Workgroups go to the 8 XCDs round-robin in dispatch order, and each XCD
// has its own L2. The blocks that read the same K/V tiles - one (head, key
// split) group, all its row tiles - are given consecutive dispatch slots of
// one XCD, so they start together there and share that L2. Within a group
// the row tiles go last to first: in a chunk the later rows see more keys,
// so the longest blocks start first and the short ones fill the last round.
// Grid: (nrt * nsplit, BH); falls back to the plain order when the groups do
// not divide evenly over the XCDs.
constexpr int kXcds = 8;
struct BlockId { int rt, sp, bh; };
__device__ __forceinline__ BlockId block_id(int nsplit) {
  const int nrt = gridDim.x / nsplit, ngroups = nsplit * gridDim.y;
  const int lin = blockIdx.x + blockIdx.y * gridDim.x;
  int grp, rt;
  if (ngroups % kXcds == 0) {
    const int i = lin / kXcds;
    grp = (i / nrt) * kXcds + lin % kXcds;
    rt = nrt - 1 - i % nrt;
  } else {
    grp = lin / nrt;
    rt = nrt - 1 - lin % nrt;
  }
  return BlockId{rt, grp % nsplit, grp / nsplit};
}

// ------------------------------------------------------------------ pass A
// Online (max, sum) update of one tile for every query of the wave. The
// running maximum m is kept in raw score units (c > 0 keeps the order);
// l sums exp2(c*(s - m)). Unmasked tiles have finite scores, so only masked
// tiles need the guard for a maximum that is still -inf.
template <int MK, int NQB>
__device__ __forceinline__ void lse_update(const f32x4 (&sacc)[2][NQB], float (&m)[NQB],
                                           float (&l)[NQB], const int (&qi)[NQB], int j0, int M,
                                           int lane, float c, const Rel& rl) {
  constexpr bool MASKED = MK == 1 || MK == 2;
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    float x[8];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float v = sacc[kb][qb][r];
        if (key_hidden<MK>(rl, kb, r, j0 + kb * 16 + 4 * (lane >> 4) + r, M, qi[qb]))
          v = -INFINITY;
        x[kb * 4 + r] = v;
      }
    const float mn = __builtin_fmaxf(__builtin_fmaxf(__builtin_fmaxf(x[0], x[1]), x[2]),
                     __builtin_fmaxf(__builtin_fmaxf(__builtin_fmaxf(x[3], x[4]), x[5]),
                                     __builtin_fmaxf(__builtin_fmaxf(x[6], x[7]), m[qb])));
    const float ms = (MASKED && mn == -INFINITY) ? 0.f : mn * c;
    float acc = l[qb] * __builtin_amdgcn_exp2f(fmaf(m[qb], c, -ms));
#pragma unroll
    for (int e = 0; e < 8; ++e) acc += __builtin_amdgcn_exp2f(fmaf(x[e], c, -ms));
    l[qb] = acc;
    m[qb] = mn;
  }
}

// Loop state of pass A. At the start of tile t: sa holds S(t), and ka (ra in
// cache mode: the relative positions) holds the global rows of tile t+2,
// loaded but not yet written to LDS; kb (rb) is free.
template <int D, int NT, int NQB>
struct LseState {
  f32x4 sa[2][NQB], sb[2][NQB];
  u32x4 ka[Tile<D, NT>::N], kb[Tile<D, NT>::N];
  int ra, rb;
};

// One tile of pass A: the loads of tile t+3 go to `fill` while the MFMAs of
// S(t+1) and the update with S(t) run; then tile t+2 (in `put`) goes to the
// LDS buffer tile t-1 used. The loads of tile t+3 are waited for only one
// tile later.
template <int MK, bool SEL, int D, int NT, int NQB>
__device__ __forceinline__ void lse_tile(int t, int t0, int t1, const f32x4 (&s_cur)[2][NQB],
                                         f32x4 (&s_nxt)[2][NQB], u32x4 (&fill)[Tile<D, NT>::N],
                                         const u32x4 (&put)[Tile<D, NT>::N], int& rfill,
                                         int rput, const Tile<D, NT>& tl,
                                         bf16_t (*Ks)[BN * kstride(D)], int (*rps)[kRpPitch],
                                         const bf16x8 (&qf)[NQB][D / 32], float (&m)[NQB],
                                         float (&l)[NQB], const int (&qi)[NQB],
                                         const bf16_t* kc_bh, const bf16_t* kn_bh,
                                         const int32_t* tp_bh, const Geo& g, int lane, float c) {
  const int b0 = (t - t0) % NBUF, b1 = (t + 1 - t0) % NBUF, b2 = (t + 2 - t0) % NBUF;
  const int jn = min(t + 3, t1 - 1) * BN;
  load_tile<D, NT>(fill, tl, kc_bh, kn_bh, jn, g.M, g.Nk);
  if (MK >= 2) rfill = load_tp(tp_bh, jn, g.M);
  Rel rl;
  if (MK == 2) load_rel(rl, rps[b0], lane);
  scores_tile<D, NQB>(s_nxt, Ks[b1], qf, lane);
  lse_update<MK, NQB>(s_cur, m, l, qi, t * BN, g.M, lane, c, rl);
  interleave<2 * NQB * (D / 32), MK ? 8 : 5>();
  store_tile<D, NT>(Ks[b2], tl.loff, put);
  if (MK >= 2) store_rp<SEL>(rps[b2], rput, g.pos0, min(t + 2, t1 - 1) * BN, g.M);
  __syncthreads();
}

// Cache mode with SEL (MK 2): a tile every row of the wave sees runs the
// body without the mask (MK 3). The choice is wave-uniform and made per
// tile, between two straight-line bodies.
template <int MK, bool SEL, int D, int NT, int NQB>
__device__ __forceinline__ void lse_tile_sel(int t, int t0, int t1, const f32x4 (&s_cur)[2][NQB],
                                             f32x4 (&s_nxt)[2][NQB],
                                             u32x4 (&fill)[Tile<D, NT>::N],
                                             const u32x4 (&put)[Tile<D, NT>::N], int& rfill,
                                             int rput, const Tile<D, NT>& tl,
                                             bf16_t (*Ks)[BN * kstride(D)],
                                             int (*rps)[kRpPitch],
                                             const bf16x8 (&qf)[NQB][D / 32], float (&m)[NQB],
                                             float (&l)[NQB], const int (&qi)[NQB],
                                             const bf16_t* kc_bh, const bf16_t* kn_bh,
                                             const int32_t* tp_bh, const Geo& g, int lane,
                                             float c) {
  if (SEL && MK == 2 && !tile_needs_mask<NQB>(rps[(t - t0) % NBUF], qi))
    lse_tile<3, SEL, D, NT, NQB>(t, t0, t1, s_cur, s_nxt, fill, put, rfill, rput, tl, Ks, rps,
                                 qf, m, l, qi, kc_bh, kn_bh, tp_bh, g, lane, c);
  else
    lse_tile<MK, SEL, D, NT, NQB>(t, t0, t1, s_cur, s_nxt, fill, put, rfill, rput, tl, Ks, rps,
                                  qf, m, l, qi, kc_bh, kn_bh, tp_bh, g, lane, c);
}

// Runs the tiles [ta, tb) of a loop in pieces by the kind of load they
// issue. The tile for t loads tile min(t+3, t1-1) ahead; a tile wholly inside
// the cache or wholly inside the chunk loads from one base row (PURE, no
// branch), while a tile holding keys of both (it starts below M and ends
// above it) or a ragged last tile needs the per-row choice. The tile that
// loads the tile across M, and the last four when tile t1-1 is ragged, run
// the general body; the rest run straight-line bodies. run(pure, a, b) runs
// tiles [a, b), with pure a std::true_type or std::false_type.
template <class F>
__device__ __forceinline__ void by_load_kind(int ta, int tb, int t1, int M, int Nk, F&& run) {
  const auto mixed = [M, Nk](int t) {
    const int j0 = t * BN;
    return (j0 < M && j0 + BN > M) || j0 + BN > Nk;
  };
  const int tm = M / BN;   // the tile across M when M is not a multiple of BN
  const int p = (tm < t1 - 1 && mixed(tm)) ? tm - 3 : INT_MAX;
  const int z = mixed(t1 - 1) ? t1 - 4 : INT_MAX;   // p < z
  int a = ta;
  const auto piece = [&](auto pure, int e) {
    e = min(e, tb);
    if (a < e) run(pure, a, e);
    a = max(a, e);
  };
  piece(std::true_type{}, min(p, z));
  if (a == p) piece(std::false_type{}, p + 1);
  piece(std::true_type{}, z);
  piece(std::false_type{}, tb);
}

// Tiles [ta, tb): two tiles per trip with the roles of the register sets
// swapped, so no accumulator or staging register is copied; an odd last
// tile restores the state invariant with one copy.
template <int MK, bool SEL, int D, int NT, int NQB>
__device__ __forceinline__ void lse_loop(int ta, int tb, int t0, int t1, LseState<D, NT, NQB>& S,
                                         const Tile<D, NT>& tl,
                                         bf16_t (*Ks)[BN * kstride(D)], int (*rps)[kRpPitch],
                                         const bf16x8 (&qf)[NQB][D / 32], float (&m)[NQB],
                                         float (&l)[NQB], const int (&qi)[NQB],
                                         const bf16_t* kc_bh, const bf16_t* kn_bh,
                                         const int32_t* tp_bh, const Geo& g, int lane, float c) {
  int t = ta;
  for (; t + 1 < tb; t += 2) {
    lse_tile_sel<MK, SEL, D, NT, NQB>(t, t0, t1, S.sa, S.sb, S.kb, S.ka, S.rb, S.ra, tl, Ks, rps,
                                      qf, m, l, qi, kc_bh, kn_bh, tp_bh, g, lane, c);
    lse_tile_sel<MK, SEL, D, NT, NQB>(t + 1, t0, t1, S.sb, S.sa, S.ka, S.kb, S.ra, S.rb, tl, Ks,
                                      rps, qf, m, l, qi, kc_bh, kn_bh, tp_bh, g, lane, c);
  }
  if (t < tb) {
    lse_tile_sel<MK, SEL, D, NT, NQB>(t, t0, t1, S.sa, S.sb, S.kb, S.ka, S.rb, S.ra, tl, Ks, rps,
                                      qf, m, l, qi, kc_bh, kn_bh, tp_bh, g, lane, c);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) S.sa[kb][qb] = S.sb[kb][qb];
#pragma unroll
    for (int e = 0; e < Tile<D, NT>::N; ++e) S.ka[e] = S.kb[e];
    S.ra = S.rb;
  }
}

// First tile index at which a row tile starting at packed row row0 needs a
// mask: in chunk mode the first tile reaching a chunk key some row cannot
// see, in cache mode (CACHE) every tile.
template <bool CACHE>
__device__ __forceinline__ int mask_start(const Geo& g, int row0, int t0, int t1) {
  if (CACHE) return t0;
  return min(t1, max(t0, first_masked_tile(g.M, min(row0, g.R - 1) / g.G)));
}

// SEL (cache mode only): tiles every row of a wave sees skip the mask.
template <int D, int NW, int NQB, bool CACHE, bool SEL>
__global__ __launch_bounds__(NW * 64) void lse_pass(Geo g, int Hq, int Hkv, int nsplit,
                                                    float c_log2, float2* __restrict__ stats) {
  constexpr int NT = NW * 64, ROWS = NW * NQB * 16;
  constexpr int MKM = CACHE ? 2 : 1;   // mask mode of the masked tiles
  __shared__ __attribute__((aligned(16))) bf16_t Ks[NBUF][BN * kstride(D)];
  __shared__ __attribute__((aligned(16))) int rps[NBUF][kRpPitch];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const BlockId id = block_id(nsplit);
  const int rt = id.rt, sp = id.sp;
  const size_t bh = id.bh;
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  const int row0 = rt * ROWS, wrow0 = row0 + wave * NQB * 16;
  const int kv_end = kv_end_for_rows(min(row0 + ROWS, g.R), g.G, g.T, g.M, g.Tk);
  int t0, t1;
  split_range((kv_end + BN - 1) / BN, nsplit, sp, t0, t1);
  const int t_mask = mask_start<CACHE>(g, row0, t0, t1);
  const bf16_t* kc_bh = g.kc + bh * (size_t)g.M * D;
  const bf16_t* kn_bh = CACHE ? nullptr : g.kn + bh * (size_t)g.T * D;
  const int32_t* tp_bh = CACHE ? g.tp + bh * (size_t)g.M : nullptr;

  bf16x8 qf[NQB][D / 32];
  load_q<D, NQB>(qf, g, b, h, Hq, wrow0, lane);
  int qi[NQB];
  float m[NQB], l[NQB];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    qi[qb] = (wrow0 + qb * 16 + (lane & 15)) / g.G;
    m[qb] = -INFINITY;
    l[qb] = 0.f;
  }

  LseState<D, NT, NQB> S;
  const Tile<D, NT> tl;
  if (t0 < t1) {
    const int j1 = min(t0 + 1, t1 - 1) * BN, j2 = min(t0 + 2, t1 - 1) * BN;
    load_tile<D, NT>(S.ka, tl, kc_bh, kn_bh, t0 * BN, g.M, g.Nk);
    load_tile<D, NT>(S.kb, tl, kc_bh, kn_bh, j1, g.M, g.Nk);
    if (CACHE) {
      store_rp<SEL>(rps[0], load_tp(tp_bh, t0 * BN, g.M), g.pos0, t0 * BN, g.M);
      store_rp<SEL>(rps[1], load_tp(tp_bh, j1, g.M), g.pos0, j1, g.M);
      S.ra = load_tp(tp_bh, j2, g.M);
    }
    store_tile<D, NT>(Ks[0], tl.loff, S.ka);
    store_tile<D, NT>(Ks[1], tl.loff, S.kb);
    load_tile<D, NT>(S.ka, tl, kc_bh, kn_bh, j2, g.M, g.Nk);
    __syncthreads();
    scores_tile<D, NQB>(S.sa, Ks[0], qf, lane);
    lse_loop<0, false, D, NT, NQB>(t0, t_mask, t0, t1, S, tl, Ks, rps, qf, m, l, qi, kc_bh,
                                   kn_bh, tp_bh, g, lane, c_log2);
    lse_loop<MKM, SEL, D, NT, NQB>(t_mask, t1, t0, t1, S, tl, Ks, rps, qf, m, l, qi, kc_bh,
                                   kn_bh, tp_bh, g, lane, c_log2);
  }
  // merge the four lane groups (disjoint key subsets of the same query)
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    m[qb] *= c_log2;                    // raw score units -> log2 units
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
// Probabilities of one tile (bf16 B operands of the PV product) and their
// column partials over this wave's rows, into the wave's LDS row for the
// tile (the four lanes holding one column's total all store it).
template <int MK, int NQB>
__device__ __forceinline__ void probs_tile(const f32x4 (&sacc)[2][NQB], bf16x8 (&pb)[NQB],
                                           const float (&lam)[NQB], const int (&qi)[NQB],
                                           float* cs_row, int j0, int M, int lane, float c,
                                           const Rel& rl) {
  float cs[2][4];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float p = __builtin_amdgcn_exp2f(fmaf(sacc[kb][qb][r], c, -lam[qb]));
        if (key_hidden<MK>(rl, kb, r, j0 + kb * 16 + 4 * (lane >> 4) + r, M, qi[qb])) p = 0.f;
        cs[kb][r] = qb == 0 ? p : cs[kb][r] + p;
        pb[qb][kb * 4 + r] = (__bf16)p;
      }
  }
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const float v = colsum16(cs[kb][0], cs[kb][1], cs[kb][2], cs[kb][3], lane);
    cs_row[kb * 16 + 4 * (lane >> 4) + ((lane & 15) >> 2)] = v;
  }
}

// O^T += V^T P^T for one tile.
template <int D, int NQB>
__device__ __forceinline__ void pv_tile(f32x4 (&oacc)[D / 16][NQB], const bf16x8 (&pb)[NQB],
                                        const bf16_t* Vs, int lane) {
#pragma unroll
  for (int db = 0; db < D / 16; ++db) {
    const bf16x8 a = v_operand<D>(Vs, db, lane);
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) oacc[db][qb] = mfma(a, pb[qb], oacc[db][qb]);
  }
}

// Loop state of pass B, with the invariant of pass A: at the start of tile t,
// sa holds S(t) and (ka, va) the rows of tile t+2 not yet in LDS.
template <int D, int NT, int NQB>
struct MainState {
  f32x4 sa[2][NQB], sb[2][NQB];
  f32x4 oacc[D / 16][NQB];
  u32x4 ka[Tile<D, NT>::N], va[Tile<D, NT>::N], kb[Tile<D, NT>::N], vb[Tile<D, NT>::N];
  int ra, rb;   // cache mode: relative positions of tile t+2 / free
};

// One tile of pass B. The waves' column partials of the tile meet in
// cs_lds[tile parity][wave]; after the tile's barrier, threads 0..BN-1 add
// them in wave order and store the block's partial row (one partial per
// block and row tile).
template <int MK, bool PURE, int D, int NT, int NQB>
__device__ __forceinline__ void main_tile(
    int t, int t0, int t1, const f32x4 (&s_cur)[2][NQB], f32x4 (&s_nxt)[2][NQB],
    f32x4 (&oacc)[D / 16][NQB], u32x4 (&kfill)[Tile<D, NT>::N],
    u32x4 (&vfill)[Tile<D, NT>::N], const u32x4 (&kput)[Tile<D, NT>::N],
    const u32x4 (&vput)[Tile<D, NT>::N], int& rfill, int rput, const Tile<D, NT>& tl,
    bf16_t (*Ks)[BN * kstride(D)], bf16_t (*Vs)[BN * vstride(D)], int (*rps)[kRpPitch],
    const bf16x8 (&qf)[NQB][D / 32], const float (&lam)[NQB], const int (&qi)[NQB],
    float (*cs_lds)[NT / 64][BN], float* prow, const bf16_t* kc_bh, const bf16_t* kn_bh,
    const bf16_t* vc_bh, const bf16_t* vn_bh, const int32_t* tp_bh, const Geo& g, int lane,
    float c) {
  const int wave = threadIdx.x >> 6;
  const int j0 = t * BN;
  const int b0 = (t - t0) % NBUF, b1 = (t + 1 - t0) % NBUF, b2 = (t + 2 - t0) % NBUF;
  const int jn = min(t + 3, t1 - 1) * BN;
  load_tile<D, NT, PURE>(kfill, tl, kc_bh, kn_bh, jn, g.M, g.Nk);
  load_tile<D, NT, PURE>(vfill, tl, vc_bh, vn_bh, jn, g.M, g.Nk);
  if (MK >= 2) rfill = load_tp(tp_bh, jn, g.M);
  Rel rl;
  if (MK == 2) load_rel(rl, rps[b0], lane);
  bf16x8 pb[NQB];
  scores_tile<D, NQB>(s_nxt, Ks[b1], qf, lane);
  probs_tile<MK, NQB>(s_cur, pb, lam, qi, cs_lds[(t - t0) & 1][wave], j0, g.M, lane, c, rl);
  pv_tile<D, NQB>(oacc, pb, Vs[b0], lane);
  interleave<2 * NQB * (D / 32), MK ? 5 : 4>();
  interleave<NQB * (D / 16), 1>();
  store_tile<D, NT>(Ks[b2], tl.loff, kput);
  store_tile<D, NT>(Vs[b2], tl.vloff, vput);
  if (MK >= 2) store_rp<false>(rps[b2], rput, g.pos0, min(t + 2, t1 - 1) * BN, g.M);
  __syncthreads();
  if (threadIdx.x < BN) {
    const float (*cs)[BN] = cs_lds[(t - t0) & 1];
    float a = cs[0][threadIdx.x];
#pragma unroll
    for (int w = 1; w < NT / 64; ++w) a += cs[w][threadIdx.x];
    prow[j0 + threadIdx.x] = a;
  }
}

// Tiles [ta, tb) of pass B, with the trip structure of pass A.
template <int MK, bool PURE, int D, int NT, int NQB>
__device__ __forceinline__ void main_loop(int ta, int tb, int t0, int t1, MainState<D, NT, NQB>& S,
                                          const Tile<D, NT>& tl,
                                          bf16_t (*Ks)[BN * kstride(D)],
                                          bf16_t (*Vs)[BN * vstride(D)], int (*rps)[kRpPitch],
                                          const bf16x8 (&qf)[NQB][D / 32],
                                          const float (&lam)[NQB], const int (&qi)[NQB],
                                          float (*cs_lds)[NT / 64][BN], float* prow,
                                          const bf16_t* kc_bh, const bf16_t* kn_bh,
                                          const bf16_t* vc_bh, const bf16_t* vn_bh,
                                          const int32_t* tp_bh, const Geo& g, int lane, float c) {
  int t = ta;
  for (; t + 1 < tb; t += 2) {
    main_tile<MK, PURE, D, NT, NQB>(t, t0, t1, S.sa, S.sb, S.oacc, S.kb, S.vb, S.ka, S.va, S.rb,
                                    S.ra, tl, Ks, Vs, rps, qf, lam, qi, cs_lds, prow, kc_bh, kn_bh,
                                    vc_bh, vn_bh, tp_bh, g, lane, c);
    main_tile<MK, PURE, D, NT, NQB>(t + 1, t0, t1, S.sb, S.sa, S.oacc, S.ka, S.va, S.kb, S.vb,
                                    S.ra, S.rb, tl, Ks, Vs, rps, qf, lam, qi, cs_lds, prow, kc_bh,
                                    kn_bh, vc_bh, vn_bh, tp_bh, g, lane, c);
  }
  if (t < tb) {
    main_tile<MK, PURE, D, NT, NQB>(t, t0, t1, S.sa, S.sb, S.oacc, S.kb, S.vb, S.ka, S.va, S.rb,
                                    S.ra, tl, Ks, Vs, rps, qf, lam, qi, cs_lds, prow, kc_bh, kn_bh,
                                    vc_bh, vn_bh, tp_bh, g, lane, c);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) S.sa[kb][qb] = S.sb[kb][qb];
#pragma unroll
    for (int e = 0; e < Tile<D, NT>::N; ++e) {
      S.ka[e] = S.kb[e];
      S.va[e] = S.vb[e];
    }
    S.ra = S.rb;
  }
}

template <int D, int NW, int NQB, bool CACHE>
__global__ __launch_bounds__(NW * 64) void main_pass(Geo g, int Hq, int Hkv, int nsplit,
                                                     int nsplit_lse, float c_log2,
                                                     const float2* __restrict__ stats,
                                                     float* __restrict__ parts, int parts_ld,
                                                     bf16_t* __restrict__ out,
                                                     float* __restrict__ opart,
                                                     float* __restrict__ lse_out) {
  constexpr int NT = NW * 64, ROWS = NW * NQB * 16;
  constexpr int MKM = CACHE ? 2 : 1;   // mask mode of the masked tiles
  __shared__ __attribute__((aligned(16))) bf16_t Ks[NBUF][BN * kstride(D)];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[NBUF][BN * vstride(D)];
  __shared__ __attribute__((aligned(16))) int rps[NBUF][kRpPitch];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const BlockId id = block_id(nsplit);
  const int rt = id.rt, sp = id.sp;
  const size_t bh = id.bh;
  const int BH = gridDim.y;
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  const int row0 = rt * ROWS, wrow0 = row0 + wave * NQB * 16;
  const int kv_end = kv_end_for_rows(min(row0 + ROWS, g.R), g.G, g.T, g.M, g.Tk);
  int t0, t1;
  split_range((kv_end + BN - 1) / BN, nsplit, sp, t0, t1);
  const int t_mask = mask_start<CACHE>(g, row0, t0, t1);
  const bf16_t* kc_bh = g.kc + bh * (size_t)g.M * D;
  const bf16_t* kn_bh = CACHE ? nullptr : g.kn + bh * (size_t)g.T * D;
  const bf16_t* vc_bh = g.vc + bh * (size_t)g.M * D;
  const bf16_t* vn_bh = CACHE ? nullptr : g.vn + bh * (size_t)g.T * D;
  const int32_t* tp_bh = CACHE ? g.tp + bh * (size_t)g.M : nullptr;

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
      for (int s = 0; s < nsplit_lse; ++s)
        mx = fmaxf(mx, stats[((size_t)s * BH + bh) * g.R + r].x);
      float L = 0.f;
      for (int s = 0; s < nsplit_lse; ++s) {
        const float2 st = stats[((size_t)s * BH + bh) * g.R + r];
        if (st.y > 0.f) L += st.y * __builtin_amdgcn_exp2f(st.x - mx);
      }
      // a row that sees no key (cache mode only) has no softmax: every
      // probability is 0 and its lse is -inf
      lam[qb] = L > 0.f ? mx + __log2f(L) : INFINITY;
    } else {
      lam[qb] = INFINITY;   // padding rows: every probability is 0
    }
    if (sp == 0 && lane < 16 && r < g.R) {
      const int i = r / g.G, gg = r % g.G;
      lse_out[(size_t)(b * Hq + h * g.G + gg) * g.T + i] =
          lam[qb] == INFINITY ? -INFINITY : lam[qb] * kLn2;
    }
  }

  MainState<D, NT, NQB> S;
#pragma unroll
  for (int db = 0; db < D / 16; ++db)
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) S.oacc[db][qb] = f32x4{0.f, 0.f, 0.f, 0.f};

  __shared__ float cs_lds[2][NW][BN];
  float* prow = parts + ((size_t)rt * BH + bh) * parts_ld;
  const Tile<D, NT> tl;

  if (t0 < t1) {
    const int j1 = min(t0 + 1, t1 - 1) * BN, j2 = min(t0 + 2, t1 - 1) * BN;
    load_tile<D, NT>(S.ka, tl, kc_bh, kn_bh, t0 * BN, g.M, g.Nk);
    load_tile<D, NT>(S.va, tl, vc_bh, vn_bh, t0 * BN, g.M, g.Nk);
    load_tile<D, NT>(S.kb, tl, kc_bh, kn_bh, j1, g.M, g.Nk);
    load_tile<D, NT>(S.vb, tl, vc_bh, vn_bh, j1, g.M, g.Nk);
    if (CACHE) {
      store_rp<false>(rps[0], load_tp(tp_bh, t0 * BN, g.M), g.pos0, t0 * BN, g.M);
      store_rp<false>(rps[1], load_tp(tp_bh, j1, g.M), g.pos0, j1, g.M);
      S.ra = load_tp(tp_bh, j2, g.M);
    }
    store_tile<D, NT>(Ks[0], tl.loff, S.ka);
    store_tile<D, NT>(Vs[0], tl.vloff, S.va);
    store_tile<D, NT>(Ks[1], tl.loff, S.kb);
    store_tile<D, NT>(Vs[1], tl.vloff, S.vb);
    load_tile<D, NT>(S.ka, tl, kc_bh, kn_bh, j2, g.M, g.Nk);
    load_tile<D, NT>(S.va, tl, vc_bh, vn_bh, j2, g.M, g.Nk);
    __syncthreads();
    scores_tile<D, NQB>(S.sa, Ks[0], qf, lane);
    by_load_kind(t0, t_mask, t1, g.M, g.Nk, [&](auto pure, int a, int e) {
      main_loop<0, decltype(pure)::value, D, NT, NQB>(a, e, t0, t1, S, tl, Ks, Vs, rps, qf, lam,
                                                      qi, cs_lds, prow, kc_bh, kn_bh, vc_bh,
                                                      vn_bh, tp_bh, g, lane, c_log2);
    });
    by_load_kind(t_mask, t1, t1, g.M, g.Nk, [&](auto pure, int a, int e) {
      main_loop<MKM, decltype(pure)::value, D, NT, NQB>(a, e, t0, t1, S, tl, Ks, Vs, rps, qf,
                                                        lam, qi, cs_lds, prow, kc_bh, kn_bh,
                                                        vc_bh, vn_bh, tp_bh, g, lane, c_log2);
    });
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
      const f32x4 o = S.oacc[db][qb];
      if (nsplit == 1) {
        uint2 v;
        v.x = (uint32_t)f32_to_bf16(o[0]) | ((uint32_t)f32_to_bf16(o[1]) << 16);
        v.y = (uint32_t)f32_to_bf16(o[2]) | ((uint32_t)f32_to_bf16(o[3]) << 16);
        *reinterpret_cast<uint2*>(out + orow + dd) = v;
      } else {
        float* dst = opart + (((size_t)sp * BH + bh) * g.R + r) * D + dd;
        *reinterpret_cast<float4*>(dst) = make_float4(o[0], o[1], o[2], o[3]);
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

// Both passes use 128-row blocks of 4 waves x 32 rows: few enough registers
// per wave that two or more waves share each SIMD and hide each other's
// latencies.
// Both passes run 128-row blocks of 4 waves x 32 rows, or at d = 128
// 256-row blocks of 8 waves where the plan finds those fill whole rounds of
// the CUs (so the waves that share a SIMD come from fewer blocks).
constexpr int kLseQB = 2, kMainQB = 2;

template <int D>
hipError_t run(const Shape& s, const Plan& p, const void* q, const void* kc, const void* vc,
               const void* kn, const void* vn, void* out, float* lse, float* wsum, char* ws,
               float scale, KeyPos kp, hipStream_t st, ScoreAcc acc) {
  const int main_waves = D == 128 && p.main_waves == 8 ? 8 : 4;
  const int ROWS = main_waves * kMainQB * 16;
  const int lse_waves = D == 128 && p.lse_waves == 8 ? 8 : 4;
  // cache mode: the lse pass skips the mask on tiles every row of a wave
  // sees where the chunk's tokens are few among the slots (most tiles hold
  // none some row cannot see), and in 8-wave blocks, whose kernel fits four
  // waves per SIMD (116 registers) only in this form (130 without it)
  const bool sel = s.cache_only && (lse_waves == 8 || (long long)s.T * 16 <= (long long)s.M);
  const int LSE_ROWS = lse_waves * kLseQB * 16;
  Geo g{s.G(), s.T, s.M, s.R(), s.Nk(), s.Tk(), (const bf16_t*)q, (const bf16_t*)kc,
        (const bf16_t*)vc, (const bf16_t*)kn, (const bf16_t*)vn, kp.tp, kp.pos0};
  const bool cache = s.cache_only;
  const int nrt = (s.R() + ROWS - 1) / ROWS, nrt_lse = (s.R() + LSE_ROWS - 1) / LSE_ROWS;
  dim3 grid(nrt * p.nsplit, s.BH()), grid_lse(nrt_lse * p.nsplit_lse, s.BH());
  const float c = scale * kLog2e;
  float2* stats = reinterpret_cast<float2*>(ws + p.off_stats);
  float* parts = reinterpret_cast<float*>(ws + p.off_parts);
  float* opart = reinterpret_cast<float*>(ws + p.off_opart);
  auto lse_k = [&](auto kern) {
    return launch_kernel(K_MFMA_LSE, kern, grid_lse, dim3(lse_waves * 64), st, g, s.Hq, s.Hkv,
                         p.nsplit_lse, c, stats);
  };
  hipError_t e;
  if constexpr (D == 128) {
    if (lse_waves == 8)
      e = !cache ? lse_k(lse_pass<D, 8, kLseQB, false, false>)
          : sel  ? lse_k(lse_pass<D, 8, kLseQB, true, true>)
                 : lse_k(lse_pass<D, 8, kLseQB, true, false>);
    else
      e = !cache ? lse_k(lse_pass<D, 4, kLseQB, false, false>)
          : sel  ? lse_k(lse_pass<D, 4, kLseQB, true, true>)
                 : lse_k(lse_pass<D, 4, kLseQB, true, false>);
  } else {
    e = !cache ? lse_k(lse_pass<D, 4, kLseQB, false, false>)
        : sel  ? lse_k(lse_pass<D, 4, kLseQB, true, true>)
               : lse_k(lse_pass<D, 4, kLseQB, true, false>);
  }
  if (e != hipSuccess) return e;
  auto main = [&](auto kern) {
    return launch_kernel(K_MFMA_MAIN, kern, grid, dim3(main_waves * 64), st, g, s.Hq, s.Hkv,
                         p.nsplit, p.nsplit_lse, c, (const float2*)stats, parts, p.parts_ld,
                         (bf16_t*)out, opart, lse);
  };
  if constexpr (D == 128) {
    if (main_waves == 8)
      e = cache ? main(main_pass<D, 8, kMainQB, true>) : main(main_pass<D, 8, kMainQB, false>);
    else
      e = cache ? main(main_pass<D, 4, kMainQB, true>) : main(main_pass<D, 4, kMainQB, false>);
  } else {
    e = cache ? main(main_pass<D, 4, kMainQB, true>) : main(main_pass<D, 4, kMainQB, false>);
  }
  if (e != hipSuccess) return e;
  if (p.nsplit > 1) {
    const size_t n4 = (size_t)s.BH() * s.R() * s.d / 4;
    e = launch_kernel(K_SPLIT_REDUCE, split_reduce<D>, dim3((unsigned)((n4 + 255) / 256)),
                      dim3(256), st, (const float*)opart, (bf16_t*)out, s.Hq, s.Hkv, s.G(), s.T,
                      s.R(), s.BH(), p.nsplit);
    if (e != hipSuccess) return e;
  }
  return launch_colsum_reduce(s, p, parts, wsum, st, acc);
}

}  // namespace

// Rows of packed queries per workgroup of the MFMA kernels, and per colsum
// partial (one partial per block).
int mfma_rows_per_wave() { return kMainQB * 16; }

hipError_t launch_sdpa_mfma(const Shape& s, const Plan& p, const void* q, const void* kc,
                            const void* vc, const void* kn, const void* vn, void* out, float* lse,
                            float* wsum, char* ws, float scale, KeyPos kp, hipStream_t st,
                            ScoreAcc acc) {
  if (s.d == 64)
    return run<64>(s, p, q, kc, vc, kn, vn, out, lse, wsum, ws, scale, kp, st, acc);
  return run<128>(s, p, q, kc, vc, kn, vn, out, lse, wsum, ws, scale, kp, st, acc);
}

}  // namespace h2o
