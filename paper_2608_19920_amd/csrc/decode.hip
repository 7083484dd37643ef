// Token generation (T = 1): the chunk is one query per query head, so the
// step streams the whole KV cache once and is bound by HBM bandwidth
// (Sec. "Sparse Attention. Key-Value Caching": N_q = 1, N_k = N_C).
//
//   split    block (split s, head bh): each of its 4 waves streams steps of 32
//            cache slots (steps s*4 + w, + 4 ns, ...). The G queries of the
//            group are the columns of bf16 MFMA products: S^T = K Q^T straight
//            from the loaded K rows, O^T += V^T P with V passed through LDS
//            and read back transposed. The split's softmax partial (m, l,
//            O-partial) per query head is written out, and so are the float32
//            logits for the column sums ([bh][g][slot]).
//   combine  block bh merges the splits with the chunk's own key (column M),
//            writes out and lse, and wsum[j] = sum_g exp2(logit_gj - lambda_g)
//            from the stored logits.
//
// In cache mode the chunk's key is already in the cache: there is no column
// M, and a slot whose token position is later than the query's (pos0) is
// masked; its stored logit is -inf.
#include "internal.h"

namespace h2o {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kCombThreads = 1024;                       // threads of a combine block
constexpr int kStep = 32;                                // cache slots per wave step
constexpr int kMaxGD = 512;                              // G * D handled by these kernels
constexpr int kMaxSplit = 64;                            // split blocks per head, at most

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

__device__ __forceinline__ f32x4 mfma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ u32x4 load16(const bf16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// Whole-wave reductions, the result in every lane: four DPP steps inside each
// 16-lane row (quad xor 1, quad xor 2, half-row mirror, row mirror: after
// them every lane holds its row's total), then two cross-row exchanges. All
// six steps are VALU operations, no LDS permutes.
//
// Cross-row exchange: v_permlane16_swap / v_permlane32_swap with x as both
// operands leave (a, b) = x of lanes (l, l ^ 16) or (l, l ^ 32), the lower
// lane first in both lanes of a pair, so a commutative combine of a and b
// gives equal bits in the two lanes.
template <bool ROW16>
__device__ __forceinline__ void xrow(uint32_t x, uint32_t& a, uint32_t& b) {
  if constexpr (ROW16) {
    const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    a = r[0];
    b = r[1];
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    a = r[0];
    b = r[1];
  }
}
template <bool ROW16>
__device__ __forceinline__ float xrow_sum(float v) {
  uint32_t a, b;
  xrow<ROW16>(__float_as_uint(v), a, b);
  return __uint_as_float(a) + __uint_as_float(b);
}
template <bool ROW16>
__device__ __forceinline__ float xrow_max(float v) {
  uint32_t a, b;
  xrow<ROW16>(__float_as_uint(v), a, b);
  return fmaxf(__uint_as_float(a), __uint_as_float(b));
}
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, true);
}
constexpr int kDppQuadXor1 = 0xB1, kDppQuadXor2 = 0x4E, kDppHalfMirror = 0x141,
              kDppMirror = 0x140;
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
  return __uint_as_float(dpp_u32<CTRL>(__float_as_uint(x)));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f32<kDppQuadXor1>(v);
  v += dpp_f32<kDppQuadXor2>(v);
  v += dpp_f32<kDppHalfMirror>(v);
  v += dpp_f32<kDppMirror>(v);
  return xrow_sum<false>(xrow_sum<true>(v));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f32<kDppQuadXor1>(v));
  v = fmaxf(v, dpp_f32<kDppQuadXor2>(v));
  v = fmaxf(v, dpp_f32<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f32<kDppMirror>(v));
  return xrow_max<false>(xrow_max<true>(v));
}
// (key, slot) lexicographic minimum over the wave.
template <int CTRL>
__device__ __forceinline__ void argmin_step_dpp(uint32_t& k, uint32_t& j) {
  const uint32_t ok = dpp_u32<CTRL>(k), oj = dpp_u32<CTRL>(j);
  if (ok < k || (ok == k && oj < j)) { k = ok; j = oj; }
}
template <bool ROW16>
__device__ __forceinline__ void argmin_step_xrow(uint32_t& k, uint32_t& j) {
  uint32_t k0, k1, j0, j1;
  xrow<ROW16>(k, k0, k1);
  xrow<ROW16>(j, j0, j1);
  const bool second = k1 < k0 || (k1 == k0 && j1 < j0);
  k = second ? k1 : k0;
  j = second ? j1 : j0;
}
__device__ __forceinline__ void wave_argmin(uint32_t& k, uint32_t& j) {
  argmin_step_dpp<kDppQuadXor1>(k, j);
  argmin_step_dpp<kDppQuadXor2>(k, j);
  argmin_step_dpp<kDppHalfMirror>(k, j);
  argmin_step_dpp<kDppMirror>(k, j);
  argmin_step_xrow<true>(k, j);
  argmin_step_xrow<false>(k, j);
}

// floats per row of the stored logits ([bh][g][slot]; 16-byte aligned rows)
__host__ __device__ constexpr int logit_pitch(int M) { return (M + 3) & ~3; }

// bf16 per LDS row of a staged V step (32 rows x D)
template <int D>
__host__ __device__ constexpr int vpitch() { return D + 16; }

// A operand of O^T = V^T P for rows d = 16*db .. 16*db+15 of V^T. Within each
// 16-lane group, ds_read_b64_tr_b16 hands lane i element i%4 of the 8-byte
// chunks addressed by lanes 4k + i/4 (k = 0..3). Lane 4k + c of group j
// addresses slot 4j + k, columns 16*db + 4c..+3, so lane i of group j ends up
// with V[4j + k][16*db + i], k = 0..3; a second read covers slots 16 + 4j + k.
// These are the slots of the P operand built from the S^T accumulators.
template <int D>
__device__ __forceinline__ bf16x8 v_operand(const bf16_t* vs, int db, int lane) {
  const int j = lane >> 4, i = lane & 15;
  const bf16_t* p = vs + (4 * j + (i >> 2)) * vpitch<D>() + 16 * db + 4 * (i & 3);
  typedef __attribute__((address_space(3))) bf16_t lds_bf16;
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)((lds_bf16*)p));
  const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_s16x4*)((lds_bf16*)(p + 16 * vpitch<D>())));
  const s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

// Streaming split kernel.
//
// Operand layouts of v_mfma_f32_16x16x32_bf16 (A: lane l holds row l%16,
// k = 8*(l/16)..+7; B: lane l holds column l%16, the same k; C: lane l holds
// rows 4*(l/16)..+3 of column l%16):
//   S^T[slot, col] = sum_d K[slot, d] Q[col, d]: A = 16 K rows as loaded from
//     global memory (lane l: slot 16*kb + l%16, d = 32*dh + 8*(l/16)..+7),
//     B = the queries, column c holding query head c % G (columns repeat the
//     G heads, so every lane has a real logit and duplicate stores write
//     equal values).
//   O^T[d, col] += sum_slot V[slot, d] P[slot, col]: the S^T accumulators of
//     the step's two 16-slot blocks, converted to bf16, are the B operand
//     (lane l: slots 16*kb + 4*(l/16) + r); A comes from v_operand.
// Each column keeps a reference maximum m, common to the 4 lanes holding the
// column; it is raised (a wave-uniform, rare branch) when a logit exceeds it
// by more than 64 in log2 units, which keeps every exp2 term below 2^64. K
// and V come in through buffer loads whose range is the head, so slots past
// the cache read as zero; they are masked, and their logit stores go to a
// sink.
//
// INS (cache mode, the insert-first step with the h2o ranking): the block
// first picks the head's evicted slot, the (score, slot)-smallest of the
// scores before the step (every block of the head finds the same one), and
// attends as if the chunk's key, value and position pos0 were already in
// that slot: the rows read from the cache are replaced in registers. Split
// block 0 also writes them into the cache and the slot into evict_idx; the
// scores are left to the combine (slot: 0 + its summed weight). Other blocks
// may read the slot while block 0 overwrites it; they never use what they
// read there.
struct InsArgs {
  const float* scores;    // [BH][M], read only here
  const bf16_t* kn;       // [BH][d] the chunk's key and value
  const bf16_t* vn;
  int32_t* evict_idx;     // [BH]
};
constexpr int kScPre = 16;   // scores per thread prefetched before the first K/V loads

template <int D, int G, bool CACHE, bool INS>
__device__ __forceinline__ void split_body(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    int Hq, int Hkv, int M, float c_log2, float* __restrict__ logits,
    float2* __restrict__ dstat, float* __restrict__ dO, float* __restrict__ sink,
    const int32_t* __restrict__ tp, int32_t pos0, InsArgs ins) {
  static_assert(!INS || CACHE, "the insert-first step runs in cache mode");
  constexpr int DH = D / 32;                 // MFMA k-chunks of a row
  constexpr int NK = 2 * DH;                 // K loads per step (two 16-slot blocks)
  constexpr int RPL = 512 / D;               // V rows per wave load
  constexpr int NV = kStep / RPL;            // V loads per step
  constexpr int VP = vpitch<D>();
  static_assert(G <= 16 && (D == 64 || D == 128), "decode shape");
  __shared__ __attribute__((aligned(16))) bf16_t vs_all[kWaves][kStep * VP];
  __shared__ float red_m[kWaves][16], red_l[kWaves][16];
  __shared__ float ored[kWaves][G][D];
  __shared__ uint32_t red_k[kWaves], red_j[kWaves];
  __shared__ int sh_slot;
  const int s = blockIdx.x, nsplit = gridDim.x;
  const size_t bh = blockIdx.y;
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 15, grp = lane >> 4;
  const int head_steps = (M + kStep - 1) / kStep;
  const int stream = s * kWaves + wave, nstreams = nsplit * kWaves;
  const int nst = stream < head_steps ? (head_steps - stream + nstreams - 1) / nstreams : 0;
  // K and V of head bh as buffer resources: rows past the cache read as zero
  const uint32_t head_bytes = (uint32_t)M * (uint32_t)(D * 2);
  const __amdgpu_buffer_rsrc_t krs = buffer_rsrc(kc + bh * (size_t)M * D, head_bytes);
  const __amdgpu_buffer_rsrc_t vrs = buffer_rsrc(vc + bh * (size_t)M * D, head_bytes);
  // cache mode: token positions of the head (slots past the cache read as 0;
  // they are masked by the slot bound)
  const __amdgpu_buffer_rsrc_t trs =
      buffer_rsrc(CACHE ? tp + bh * (size_t)M : tp, CACHE ? (uint32_t)M * 4u : 0u);
  bf16_t* vs = vs_all[wave];
  const int vrow = lane / (D / 8), vcol = 8 * (lane % (D / 8));
  const uint32_t koff = (uint32_t)(col * D + 8 * grp) * 2u;   // + block / chunk offsets
  const uint32_t voff = (uint32_t)(vrow * D + vcol) * 2u;
  // logits are stored head-major, [bh][g][slot] with the row padded to a multiple of 4
  float* lg_out = logits + (bh * G + col % G) * (size_t)logit_pitch(M);

  // Two ring slots: a step's loads are issued before the previous step is
  // consumed, so every wait leaves the other slot's loads in flight. Steps
  // past the head read as zero (buffer range) and are masked.
  u32x4 kr[2][NK], vr[2][NV];
  int32_t tr[2][8];
  auto issue = [&](int k, int u) {
    const uint32_t base = (uint32_t)((stream + k * nstreams) * kStep) * (uint32_t)(D * 2);
    if (CACHE) {   // this lane's 8 slots: 4 consecutive ones per 16-slot block
      const uint32_t tb = (uint32_t)((stream + k * nstreams) * kStep + 4 * grp) * 4u;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        tr[u][i] = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(
            trs, (int)(tb + 64u * (i >> 2) + 4u * (i & 3)), 0, 0);
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int dh = 0; dh < DH; ++dh)
        kr[u][kb * DH + dh] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                       krs, (int)(base + koff + (uint32_t)((16 * kb * D + 32 * dh) * 2)), 0, 0));
#pragma unroll
    for (int t = 0; t < NV; ++t)
      vr[u][t] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                     vrs, (int)(base + voff + (uint32_t)(t * RPL * D * 2)), 0, 0));
  };

  bf16x8 qb[DH];
  {
    const bf16_t* qrow = q + (size_t)(b * Hq + h * G + col % G) * D + 8 * grp;
#pragma unroll
    for (int dh = 0; dh < DH; ++dh) qb[dh] = __builtin_bit_cast(bf16x8, load16(qrow + 32 * dh));
  }
  float m = -INFINITY, l = 0.f;
  f32x4 oacc[D / 16];
#pragma unroll
  for (int db = 0; db < D / 16; ++db) oacc[db] = f32x4{0.f, 0.f, 0.f, 0.f};

  int slot = -1;                                // INS: the head's evicted slot
  u32x4 knr[DH], vnr = u32x4{0u, 0u, 0u, 0u};   // INS: this lane's parts of the chunk's K, V rows
  auto consume = [&](int k, int u) {
    const int key0 = (stream + k * nstreams) * kStep;
    if (INS && (unsigned)(slot - key0) < (unsigned)kStep) {   // wave-uniform, one step per head
      const int rs = slot - key0;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        if (16 * kb + col == rs) {
#pragma unroll
          for (int dh = 0; dh < DH; ++dh) kr[u][kb * DH + dh] = knr[dh];
        }
#pragma unroll
      for (int t = 0; t < NV; ++t)
        if (t * RPL + vrow == rs) vr[u][t] = vnr;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (16 * (i >> 2) + 4 * grp + (i & 3) == rs) tr[u][i] = pos0;
    }
#pragma unroll
    for (int t = 0; t < NV; ++t)
      *reinterpret_cast<u32x4*>(vs + (t * RPL + vrow) * VP + vcol) = vr[u][t];
    f32x4 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      sacc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int dh = 0; dh < DH; ++dh)
        sacc[kb] = mfma(__builtin_bit_cast(bf16x8, kr[u][kb * DH + dh]), qb[dh], sacc[kb]);
    }
    float lg[8];
    float mx = -INFINITY;
    // wave-uniform: a step reaching past the cache (the ragged last one, or
    // a padding step), whose zero rows must not raise the reference maximum
    const bool tail = key0 + kStep > M;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      lg[i] = sacc[i >> 2][i & 3] * c_log2;
      const int key = key0 + 16 * (i >> 2) + 4 * grp + (i & 3);
      if (CACHE) {
        if (key >= M || !pos_visible(tr[u][i], pos0, 0)) lg[i] = -INFINITY;
      } else if (tail && key >= M) {
        lg[i] = -INFINITY;
      }
      mx = fmaxf(mx, lg[i]);
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {   // 4 consecutive slots of one head per lane
      // stores of masked slots go to the sink, so that no store is conditional
      const int k4 = key0 + 16 * kb + 4 * grp;
      float* dst = k4 < M ? lg_out + k4 : sink + 4 * lane;
      *reinterpret_cast<f32x4*>(dst) =
          f32x4{lg[4 * kb], lg[4 * kb + 1], lg[4 * kb + 2], lg[4 * kb + 3]};
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    if (__builtin_amdgcn_ballot_w64(mx > m + 64.f)) {    // wave-uniform, rare after the start
      const bool up = mx > m + 64.f;
      const float sc = up ? __builtin_amdgcn_exp2f(m - mx) : 1.f;
      l *= sc;
#pragma unroll
      for (int db = 0; db < D / 16; ++db) oacc[db] *= sc;
      m = up ? mx : m;
    }
    bf16x8 pb;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int key = key0 + 16 * (i >> 2) + 4 * grp + (i & 3);
      const float p = key < M && (!CACHE || lg[i] > -INFINITY)
                          ? __builtin_amdgcn_exp2f(lg[i] - m) : 0.f;
      l += p;
      pb[i] = (__bf16)p;
    }
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int db = 0; db < D / 16; ++db) oacc[db] = mfma(v_operand<D>(vs, db, lane), pb, oacc[db]);
  };

  // INS: the scores and the chunk's rows are requested before the first K/V
  // loads, so the choice of the slot waits for them alone
  float scp[INS ? kScPre : 1];
  if (INS) {
    const float* sc_bh = ins.scores + bh * (size_t)M;
#pragma unroll
    for (int u = 0; u < kScPre; ++u) {
      const int j = tid + u * kThreads;
      scp[u] = j < M ? sc_bh[j] : 0.f;
    }
#pragma unroll
    for (int dh = 0; dh < DH; ++dh) knr[dh] = load16(ins.kn + bh * (size_t)D + 32 * dh + 8 * grp);
    vnr = load16(ins.vn + bh * (size_t)D + vcol);
  }
  issue(0, 0);
  if (INS) {
    // (key, slot)-smallest, slots visited in increasing order per thread so
    // that a strict < keeps the lowest slot among equal keys; the start
    // (max key, slot 0) is a real pair whenever every key is the maximum
    uint32_t bk = 0xFFFFFFFFu, bj = 0u;
#pragma unroll
    for (int u = 0; u < kScPre; ++u) {
      const int j = tid + u * kThreads;
      const uint32_t key = order_key(scp[u]);
      if (j < M && key < bk) { bk = key; bj = (uint32_t)j; }
    }
    for (int j = tid + kScPre * kThreads; j < M; j += kThreads) {
      const uint32_t key = order_key(ins.scores[bh * (size_t)M + j]);
      if (key < bk) { bk = key; bj = (uint32_t)j; }
    }
    wave_argmin(bk, bj);
    if (lane == 0) { red_k[wave] = bk; red_j[wave] = bj; }
    __syncthreads();
    if (tid == 0) {
      for (int w = 1; w < kWaves; ++w)
        if (red_k[w] < bk || (red_k[w] == bk && red_j[w] < bj)) { bk = red_k[w]; bj = red_j[w]; }
      sh_slot = (int)bj;
    }
    __syncthreads();
    slot = sh_slot;
    if (s == 0) {   // one block per head writes the insert
      if (tid == 0) {
        ins.evict_idx[bh] = slot;
        const_cast<int32_t*>(tp)[bh * (size_t)M + slot] = pos0;
      }
      if (tid < D / 8) {
        const size_t o = (bh * (size_t)M + slot) * D + 8 * tid;
        *reinterpret_cast<u32x4*>(const_cast<bf16_t*>(kc) + o) = load16(ins.kn + bh * (size_t)D + 8 * tid);
        *reinterpret_cast<u32x4*>(const_cast<bf16_t*>(vc) + o) = load16(ins.vn + bh * (size_t)D + 8 * tid);
      }
    }
  }
  // Without token positions the loop runs whole trips of two steps: with an
  // odd count the last trip's second step lies past the head (zero rows,
  // every key masked) and changes nothing. An exit between the two halves
  // makes the compiler wait for the other ring slot's loads at the top of
  // every trip, and so does a use of a step's data scheduled above the next
  // step's loads (the scheduling barriers). The cache-mode kernels, which
  // run at fewer waves per SIMD, measured faster with the exit.
  for (int k = 0; k < nst; k += 2) {
    issue(k + 1, 1);
    if (!CACHE) __builtin_amdgcn_sched_barrier(0);
    consume(k, 0);
    if (CACHE && k + 1 >= nst) break;
    issue(k + 2, 0);
    if (!CACHE) __builtin_amdgcn_sched_barrier(0);
    consume(k + 1, 1);
  }
  // block merge, one barrier: every wave leaves its column statistics and
  // its unscaled O accumulators; then per head the common maximum over the
  // waves, each wave's weight, and the sums in wave order
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  if (grp == 0) {
    red_m[wave][col] = m;
    red_l[wave][col] = l;
  }
  if (col < G) {
#pragma unroll
    for (int db = 0; db < D / 16; ++db)
#pragma unroll
      for (int r = 0; r < 4; ++r) ored[wave][col][16 * db + 4 * grp + r] = oacc[db][r];
  }
  __syncthreads();
  for (int c = tid; c < G * D; c += kThreads) {
    const int g = c / D;
    float mg = red_m[0][g];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) mg = fmaxf(mg, red_m[w][g]);
    float a = 0.f, lt = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float mw = red_m[w][g];
      const float sw = mw == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw - mg);
      a += ored[w][g][c % D] * sw;
      lt += red_l[w][g] * sw;
    }
    dO[(bh * nsplit + s) * (size_t)(G * D) + c] = a;
    if (c % D == 0) dstat[(bh * nsplit + s) * G + g] = make_float2(mg, lt);
  }
}

// Register budgets at d = 64, where the kernels fit them without spilling:
// four waves per SIMD (128 registers) without token positions, three for the
// insert-first kernel. Cache mode, and d = 128, keep the compiler's own.
#define H2O_SPLIT_PARAMS                                                                     \
  const bf16_t *__restrict__ q, const bf16_t *__restrict__ kc, const bf16_t *__restrict__ vc, \
      int Hq, int Hkv, int M, float c_log2, float *__restrict__ logits,                       \
      float2 *__restrict__ dstat, float *__restrict__ dO, float *__restrict__ sink,           \
      const int32_t *__restrict__ tp, int32_t pos0, InsArgs ins
template <int D, int G>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(D == 64 ? 4 : 1)))
void decode_split(H2O_SPLIT_PARAMS) {
  split_body<D, G, false, false>(q, kc, vc, Hq, Hkv, M, c_log2, logits, dstat, dO, sink, tp,
                                 pos0, ins);
}
template <int D, int G>
__global__ __launch_bounds__(kThreads) void decode_split_cache(H2O_SPLIT_PARAMS) {
  split_body<D, G, true, false>(q, kc, vc, Hq, Hkv, M, c_log2, logits, dstat, dO, sink, tp, pos0,
                                ins);
}
template <int D, int G>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(D == 64 ? 3 : 1)))
void decode_split_ins(H2O_SPLIT_PARAMS) {
  split_body<D, G, true, true>(q, kc, vc, Hq, Hkv, M, c_log2, logits, dstat, dO, sink, tp, pos0,
                               ins);
}
#undef H2O_SPLIT_PARAMS

template <int D, int G, bool CACHE, bool INS>
const void* split_kernel() {
  if constexpr (INS) return reinterpret_cast<const void*>(decode_split_ins<D, G>);
  else if constexpr (CACHE) return reinterpret_cast<const void*>(decode_split_cache<D, G>);
  else return reinterpret_cast<const void*>(decode_split<D, G>);
}

// ------------------------------------------------------------------ combine
// Per-head merge of the split partials with the chunk's own key (column M),
// shared by the combine kernel and the fused finish kernel so that both give
// the same bits.
constexpr int kMaxG = kMaxGD / 64;
struct HeadStats {
  float lnew[kMaxG], lam[kMaxG], mfin[kMaxG], linv[kMaxG];
  float wt[kMaxSplit * kMaxG];   // weight of split s, head g: exp2(m_sg - mfin_g) or 0
};

// One wave per query head g: the chunk key's logit (log2 units), the common
// maximum mfin over it and the splits' maxima, lam = log2 of the softmax
// normaliser, 1 / normaliser and each split's weight, with wave reductions
// (lane s holds split s; at most 64 splits). Writes lse when asked. Ends
// synced.
// Without the chunk key (cache mode, has_chunk false) lnew is -inf, and a
// query that sees no slot gets lam = +inf (every weight 0), linv = 0 and
// lse = -inf.
// The loads (head_stats_load, for wave g < G) and the arithmetic
// (head_stats_from) are separate so that a latency-bound kernel can issue the
// loads together with its other early loads.
template <int D>
struct StatIn {
  float2 st;                         // split `lane`'s (max, sum) of query head g
  bf16_t qv[(D + 63) / 64], kv[(D + 63) / 64];   // elements lane, lane + 64 of q and k_new
};
template <int D>
__device__ __forceinline__ void head_stats_load(StatIn<D>& in, const bf16_t* q, const bf16_t* kn,
                                                const float2* dstat, int Hq, int Hkv, int G,
                                                int nsplit, size_t bh, bool has_chunk) {
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  const int lane = threadIdx.x & 63, g = threadIdx.x >> 6;
  in.st = lane < nsplit ? dstat[(bh * nsplit + lane) * G + g] : make_float2(-INFINITY, 0.f);
#pragma unroll
  for (int i = 0; i < (D + 63) / 64; ++i) {
    const int dd = lane + 64 * i;
    in.qv[i] = has_chunk && dd < D ? q[(size_t)(b * Hq + h * G + g) * D + dd] : (bf16_t)0;
    in.kv[i] = has_chunk && dd < D ? kn[bh * D + dd] : (bf16_t)0;
  }
}
template <int D, int NT>
__device__ __forceinline__ void head_stats_from(HeadStats& hs, const StatIn<D>& in, int Hq,
                                                int Hkv, int G, int nsplit, float c_log2,
                                                size_t bh, float* lse, bool has_chunk) {
  static_assert(NT / 64 >= kMaxG, "one wave per query head of the group");
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  const int lane = threadIdx.x & 63, g = threadIdx.x >> 6;
  if (g < G) {
    const float2 st = in.st;
    float lnew = -INFINITY;
    if (has_chunk) {
      float a = 0.f;
#pragma unroll
      for (int i = 0; i < (D + 63) / 64; ++i)
        if (lane + 64 * i < D) a = fmaf(bf16_to_f32(in.qv[i]), bf16_to_f32(in.kv[i]), a);
      a = wave_sum(a);
      lnew = a * c_log2;
    }
    float mx = fmaxf(lnew, st.x);
    mx = wave_max(mx);
    const float wt = st.y > 0.f ? __builtin_amdgcn_exp2f(st.x - mx) : 0.f;
    float L = st.y * wt;
    L = wave_sum(L);
    if (has_chunk) L += __builtin_amdgcn_exp2f(lnew - mx);
    if (lane < nsplit) hs.wt[lane * G + g] = wt;
    if (lane == 0) {
      const bool any = L > 0.f;
      const float lm = any ? mx + __log2f(L) : INFINITY;
      hs.lnew[g] = lnew;
      hs.lam[g] = lm;
      hs.mfin[g] = mx;
      hs.linv[g] = any ? 1.f / L : 0.f;
      if (lse) lse[(size_t)(b * Hq + h * G + g)] = any ? lm * kLn2 : -INFINITY;
    }
  }
  __syncthreads();
}
template <int D, int NT>
__device__ __forceinline__ void head_stats(HeadStats& hs, const bf16_t* q, const bf16_t* kn,
                                           const float2* dstat, int Hq, int Hkv, int G,
                                           int nsplit, float c_log2, size_t bh, float* lse,
                                           bool has_chunk = true) {
  StatIn<D> in;
  if ((int)(threadIdx.x >> 6) < G)
    head_stats_load<D>(in, q, kn, dstat, Hq, Hkv, G, nsplit, bh, has_chunk);
  head_stats_from<D, NT>(hs, in, Hq, Hkv, G, nsplit, c_log2, bh, lse, has_chunk);
}

// Output element c = g*D + dd of head bh: the chunk key's term plus the
// weighted split O-partials in split order, normalised. The first PRE
// partials come from pre[] (registers), the rest from dO.
template <int D, int PRE>
__device__ __forceinline__ float out_elem(const HeadStats& hs, const bf16_t* vn,
                                          const float* dO, const float* pre, int G,
                                          int nsplit, size_t bh, int c) {
  const int g = c / D, dd = c % D;
  float a = vn ? __builtin_amdgcn_exp2f(hs.lnew[g] - hs.mfin[g]) * bf16_to_f32(vn[bh * D + dd])
               : 0.f;
#pragma unroll
  for (int s = 0; s < PRE; ++s)
    if (s < nsplit) a = fmaf(pre[s], hs.wt[s * G + g], a);
  for (int s = PRE; s < nsplit; ++s)
    a = fmaf(dO[(bh * nsplit + s) * (size_t)(G * D) + c], hs.wt[s * G + g], a);
  return a * hs.linv[g];
}

// out rows of the G query heads of head bh from the split O-partials.
template <int D, int NT>
__device__ __forceinline__ void head_out(const HeadStats& hs, const bf16_t* vn, const float* dO,
                                         bf16_t* out, int Hq, int Hkv, int G, int nsplit,
                                         size_t bh) {
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  for (int c = threadIdx.x; c < G * D; c += NT) {
    const float v = out_elem<D, 0>(hs, vn, dO, nullptr, G, nsplit, bh, c);
    out[(size_t)(b * Hq + h * G) * D + c] = f32_to_bf16(v);
  }
}

// Summed weight of cache slot j: sum_g exp2(logit_gj - lam_g), g in order.
__device__ __forceinline__ float slot_weight(const HeadStats& hs, const float* lgb, int pitch,
                                             int G, int j) {
  float a = 0.f;
  for (int g = 0; g < G; ++g) a += __builtin_amdgcn_exp2f(lgb[(size_t)g * pitch + j] - hs.lam[g]);
  return a;
}
__device__ __forceinline__ float chunk_weight(const HeadStats& hs, int G) {
  float a = 0.f;
  for (int g = 0; g < G; ++g) a += __builtin_amdgcn_exp2f(hs.lnew[g] - hs.lam[g]);
  return a;
}

// Block (x, bh) writes wsum for columns [x*kCols, +kCols) of head bh; block
// x == 0 also writes out, lse and the chunk key's column (chunk mode: kn and
// vn non-null, wsum rows of M + 1; cache mode: both null, rows of M). With
// wsum null only out and lse are written (grid x = 1).
constexpr int kCols = 1024;

// With scores non-null (cache mode only) it also adds each slot's summed
// weight to its score: scores[j] += wsum[j], one float32 addition; with
// ins_idx non-null the head's slot ins_idx[bh] (just inserted, by the fused
// insert-first split) takes 0 + wsum[j] instead.
template <int D>
__global__ __launch_bounds__(kCombThreads) void decode_combine(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ kn, const bf16_t* __restrict__ vn,
    int Hq, int Hkv, int M, int nsplit, float c_log2, const float* __restrict__ logits,
    const float2* __restrict__ dstat, const float* __restrict__ dO, bf16_t* __restrict__ out,
    float* __restrict__ lse, float* __restrict__ wsum, float* __restrict__ scores,
    const int32_t* __restrict__ ins_idx) {
  __shared__ HeadStats hs;
  const int G = Hq / Hkv;
  const size_t bh = blockIdx.y;
  const bool has_chunk = kn != nullptr;
  head_stats<D, kCombThreads>(hs, q, kn, dstat, Hq, Hkv, G, nsplit, c_log2, bh,
                          blockIdx.x == 0 ? lse : nullptr, has_chunk);
  if (blockIdx.x == 0) head_out<D, kCombThreads>(hs, vn, dO, out, Hq, Hkv, G, nsplit, bh);
  if (!wsum) return;   // out and lse only (the attend half of a step)
  float* w = wsum + bh * (size_t)(M + (has_chunk ? 1 : 0));
  const float* lgb = logits + bh * (size_t)G * logit_pitch(M);
  const int c0 = blockIdx.x * kCols, c1 = min(M, c0 + kCols);
  float* sc = scores ? scores + bh * (size_t)M : nullptr;
  const int ins = ins_idx ? ins_idx[bh] : -1;
  for (int j = c0 + threadIdx.x; j < c1; j += kCombThreads) {
    const float wj = slot_weight(hs, lgb, logit_pitch(M), G, j);
    w[j] = wj;
    if (sc) sc[j] = (j == ins ? 0.f : sc[j]) + wj;
  }
  if (has_chunk && blockIdx.x == 0 && threadIdx.x == 0) w[M] = chunk_weight(hs, G);
}

// Fused end of a token step, one block per head: the combine above, then
// scores[j] += wsum[j] for every cache slot, the (score, slot)-smallest slot
// (lower slot first among equal scores; -0 equals +0), and the insert of the
// chunk's key, value, score wsum[M] and token position into that slot. Same
// arithmetic as the combine, accumulate and argmin-insert kernels. The block
// is latency-bound on 64 or so CUs: everything it reads (the logits and
// scores of the first pass of slots, 16 bytes per load, the split
// statistics and O-partials, the query and the chunk's key and value rows)
// is requested before the first value is used; slot groups past the cache
// do no arithmetic; and of the last pass (the only pass at the decode
// shapes) the summed weights are stored before the block's argmin, the
// scores only after the slot is chosen, so that the chosen slot's score is
// written once, with its new value.
constexpr int kFinThreads = 1024;
constexpr int kFinVec = 4;                          // consecutive slots per thread and pass
constexpr int kFinPass = kFinThreads * kFinVec;     // slots per pass

__device__ __forceinline__ bool lex_less(uint32_t ka, uint32_t ja, uint32_t kb, uint32_t jb) {
  return ka < kb || (ka == kb && ja < jb);
}

// With OUT false the block skips out and lse (written by decode_combine in
// an attend call): the eviction half of the step.
template <int D, int G, bool OUT>
__global__ __launch_bounds__(kFinThreads) void decode_finish(
    const bf16_t* __restrict__ q, bf16_t* __restrict__ kc, bf16_t* __restrict__ vc,
    const bf16_t* __restrict__ kn, const bf16_t* __restrict__ vn, int Hq, int Hkv, int M,
    int nsplit, float c_log2, const float* __restrict__ logits, const float2* __restrict__ dstat,
    const float* __restrict__ dO, bf16_t* __restrict__ out, float* __restrict__ lse,
    float* __restrict__ wsum, float* __restrict__ scores, int32_t* __restrict__ token_pos,
    int32_t* __restrict__ evict_idx, int32_t pos0) {
  constexpr int NT = kFinThreads;
  __shared__ HeadStats hs;
  __shared__ uint32_t red_k[NT / 64], red_j[NT / 64];
  const size_t bh = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int pitch = logit_pitch(M);
  float* w = wsum + bh * (size_t)(M + 1);
  float* sc = scores + bh * (size_t)M;
  const float* lgb = logits + bh * (size_t)G * pitch;
  const bool sc16 = (M & 3) == 0;     // score rows start 16-byte aligned
  // This thread's slots of a pass are j0 .. j0 + 3, j0 = base + 4 * tid. A
  // logit row is padded to a multiple of 4 slots, so a group that starts in
  // the cache is read whole; its slots past the cache are not used.
  f32x4 lg[G], sv;
  auto load_pass = [&](int base) {
    const int j0 = base + kFinVec * tid;
    if (j0 < M) {
#pragma unroll
      for (int g = 0; g < G; ++g)
        lg[g] = *reinterpret_cast<const f32x4*>(lgb + (size_t)g * pitch + j0);
      if (sc16) {
        sv = *reinterpret_cast<const f32x4*>(sc + j0);
      } else {
#pragma unroll
        for (int r = 0; r < kFinVec; ++r) sv[r] = sc[min(j0 + r, M - 1)];
      }
    }
  };
  typedef uint32_t u4 __attribute__((ext_vector_type(4)));
  u4 krow = {0u, 0u, 0u, 0u}, vrow = {0u, 0u, 0u, 0u};
  if (tid < D / 8) {
    krow = reinterpret_cast<const u4*>(kn + bh * (size_t)D)[tid];
    vrow = reinterpret_cast<const u4*>(vn + bh * (size_t)D)[tid];
  }
  // thread c < G*D owns output element c (G*D <= NT); its first kPre split
  // partials come in with the other early loads, and so do the inputs of
  // the head statistics
  constexpr int kPre = 16;
  float pre[kPre];
  const bool has_c = OUT && tid < G * D;
#pragma unroll
  for (int s = 0; s < kPre; ++s)
    pre[s] = has_c && s < nsplit ? dO[(bh * nsplit + s) * (size_t)(G * D) + tid] : 0.f;
  StatIn<D> sin;
  if (wave < G) head_stats_load<D>(sin, q, kn, dstat, Hq, Hkv, G, nsplit, bh, true);
  load_pass(0);
  head_stats_from<D, NT>(hs, sin, Hq, Hkv, G, nsplit, c_log2, bh, OUT ? lse : nullptr, true);
  if (has_c) {
    const float v = out_elem<D, kPre>(hs, vn, dO, pre, G, nsplit, bh, tid);
    const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
    out[(size_t)(b * Hq + h * G) * D + tid] = f32_to_bf16(v);
  }
  // Passes in increasing slot order; a thread visits its slots in
  // increasing order, so a strict < keeps the lowest slot among equal keys.
  // The start (max key, slot 0) is a real pair whenever every key is the
  // maximum, so the choice is always a slot of the cache.
  uint32_t bk = 0xFFFFFFFFu, bj = 0u;
  f32x4 wv, sa;
  int base = 0;
  for (;;) {
    const int j0 = base + kFinVec * tid;
    if (j0 < M) {
#pragma unroll
      for (int r = 0; r < kFinVec; ++r) {
        float wj = 0.f;
#pragma unroll
        for (int g = 0; g < G; ++g) wj += __builtin_amdgcn_exp2f(lg[g][r] - hs.lam[g]);
        wv[r] = wj;
        sa[r] = sv[r] + wj;
        const uint32_t key = order_key(sa[r]);
        if (j0 + r < M && key < bk) { bk = key; bj = (uint32_t)(j0 + r); }
      }
    }
    if (base + kFinPass >= M) break;   // the last pass is stored after the choice
#pragma unroll
    for (int r = 0; r < kFinVec; ++r)
      if (j0 + r < M) {
        w[j0 + r] = wv[r];
        sc[j0 + r] = sa[r];
      }
    base += kFinPass;
    load_pass(base);
  }
  {
    // the last pass's summed weights do not wait for the choice: stored
    // before the block's argmin, they drain while it runs
    const int j0 = base + kFinVec * tid;
#pragma unroll
    for (int r = 0; r < kFinVec; ++r)
      if (j0 + r < M) w[j0 + r] = wv[r];
  }
  wave_argmin(bk, bj);
  if (lane == 0) { red_k[wave] = bk; red_j[wave] = bj; }
  __syncthreads();
  bk = red_k[0];
  bj = red_j[0];
#pragma unroll
  for (int v = 1; v < NT / 64; ++v)
    if (lex_less(red_k[v], red_j[v], bk, bj)) { bk = red_k[v]; bj = red_j[v]; }
  const int slot = (int)bj;
  const float wnew = chunk_weight(hs, G);
  {
    const int j0 = base + kFinVec * tid;
#pragma unroll
    for (int r = 0; r < kFinVec; ++r)
      if (j0 + r == slot) sa[r] = wnew;
    if (sc16 && j0 < M) {
      *reinterpret_cast<f32x4*>(sc + j0) = sa;
    } else {
#pragma unroll
      for (int r = 0; r < kFinVec; ++r)
        if (j0 + r < M) sc[j0 + r] = sa[r];
    }
  }
  if (slot < base) {
    // (more than one pass) the slot's accumulated score was stored with an
    // earlier pass: every thread's stores complete before it is replaced
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (tid == 0) sc[slot] = wnew;
  }
  if (tid == 0) {
    w[M] = wnew;
    evict_idx[bh] = slot;
    if (token_pos) token_pos[bh * M + slot] = pos0;
  }
  if (tid < D / 8) {
    reinterpret_cast<u4*>(kc + (bh * M + slot) * (size_t)D)[tid] = krow;
    reinterpret_cast<u4*>(vc + (bh * M + slot) * (size_t)D)[tid] = vrow;
  }
}

// Split blocks per head such that all blocks of the grid are resident at
// once (blocks per CU of this kernel instance x CUs), at most kMaxSplit and
// at most one wave per step of slots.
template <int D, int G, bool CACHE, bool INS = false>
int split_count(int M, int BH) {
  static int resident = 0;
  if (!resident) {
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, split_kernel<D, G, CACHE, INS>(),
                                                     kThreads, 0) != hipSuccess || per_cu < 1)
      per_cu = 2;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus < 1)
      cus = 256;
    (void)hipGetLastError();
    resident = per_cu * cus;
  }
  int ns = resident / BH;
  const int steps = (M + kStep - 1) / kStep;
  const int max_ns = (steps + kWaves - 1) / kWaves;
  if (ns > max_ns) ns = max_ns;
  if (ns > kMaxSplit) ns = kMaxSplit;
  return ns < 1 ? 1 : ns;
}

// ins.scores non-null: the fused insert-first form (cache mode).
template <int D, int G>
hipError_t launch_split(hipStream_t st, int BH, const void* q, const void* kc, const void* vc,
                        int Hq, int Hkv, int M, float c, float* logits, float2* dstat, float* dO,
                        float* sink, KeyPos kp, int* ns, InsArgs ins) {
  if (kp.tp && ins.scores) {
    *ns = split_count<D, G, true, true>(M, BH);
    return launch_kernel(K_DECODE_SPLIT, decode_split_ins<D, G>, dim3(*ns, BH),
                         dim3(kThreads), st, (const bf16_t*)q, (const bf16_t*)kc,
                         (const bf16_t*)vc, Hq, Hkv, M, c, logits, dstat, dO, sink, kp.tp,
                         kp.pos0, ins);
  }
  if (kp.tp) {
    *ns = split_count<D, G, true>(M, BH);
    return launch_kernel(K_DECODE_SPLIT, decode_split_cache<D, G>, dim3(*ns, BH),
                         dim3(kThreads), st, (const bf16_t*)q, (const bf16_t*)kc,
                         (const bf16_t*)vc, Hq, Hkv, M, c, logits, dstat, dO, sink, kp.tp,
                         kp.pos0, ins);
  }
  *ns = split_count<D, G, false>(M, BH);
  return launch_kernel(K_DECODE_SPLIT, decode_split<D, G>, dim3(*ns, BH), dim3(kThreads),
                       st, (const bf16_t*)q, (const bf16_t*)kc, (const bf16_t*)vc, Hq, Hkv, M, c,
                       logits, dstat, dO, sink, (const int32_t*)nullptr, (int32_t)0, ins);
}

}  // namespace

int decode_max_split() { return kMaxSplit; }

// The decode kernels are instantiated for these (d, G) pairs.
bool decode_supports(int d, int G) {
  return (d == 64 && (G == 1 || G == 2 || G == 4 || G == 8)) ||
         (d == 128 && (G == 1 || G == 2 || G == 4));
}

namespace {

// The split kernel over the cache (if any); returns the split count in *ns.
hipError_t launch_decode_split(const Shape& s, const Plan& p, const void* q, const void* kc,
                               const void* vc, char* ws, float c, KeyPos kp, hipStream_t st,
                               int* ns, InsArgs ins = InsArgs{nullptr, nullptr, nullptr, nullptr}) {
  float* logits = reinterpret_cast<float*>(ws + p.off_logits);
  float2* dstat = reinterpret_cast<float2*>(ws + p.off_stats);
  float* dO = reinterpret_cast<float*>(ws + p.off_opart);
  float* sink = reinterpret_cast<float*>(ws + p.off_parts);
  *ns = 0;
  if (s.M == 0) return hipSuccess;
  const int G = s.G();
  hipError_t e = hipErrorInvalidValue;
#define H2O_SPLIT(DD, GG) \
  e = launch_split<DD, GG>(st, s.BH(), q, kc, vc, s.Hq, s.Hkv, s.M, c, logits, dstat, dO, sink, \
                           kp, ns, ins)
  if (s.d == 64) {
    if (G == 1) H2O_SPLIT(64, 1);
    else if (G == 2) H2O_SPLIT(64, 2);
    else if (G == 4) H2O_SPLIT(64, 4);
    else if (G == 8) H2O_SPLIT(64, 8);
  } else {
    if (G == 1) H2O_SPLIT(128, 1);
    else if (G == 2) H2O_SPLIT(128, 2);
    else if (G == 4) H2O_SPLIT(128, 4);
  }
#undef H2O_SPLIT
  return e;
}

}  // namespace

hipError_t launch_sdpa_decode(const Shape& s, const Plan& p, const void* q, const void* kc,
                              const void* vc, const void* kn, const void* vn, void* out,
                              float* lse, float* wsum, char* ws, float scale, KeyPos kp,
                              hipStream_t st, float* scores_acc) {
  const float c = scale * kLog2e;
  int ns = 0;
  hipError_t e = launch_decode_split(s, p, q, kc, vc, ws, c, kp, st, &ns);
  if (e != hipSuccess) return e;
  const dim3 cgrid(s.M > 0 ? (s.M + kCols - 1) / kCols : 1, s.BH());
  auto combine = s.d == 64 ? decode_combine<64> : decode_combine<128>;
  const bool chunk = !s.cache_only;
  return launch_kernel(K_DECODE_COMBINE, combine, cgrid, dim3(kCombThreads), st, (const bf16_t*)q,
                       chunk ? (const bf16_t*)kn : nullptr, chunk ? (const bf16_t*)vn : nullptr,
                       s.Hq, s.Hkv, s.M, ns, c,
                       (const float*)(ws + p.off_logits), (const float2*)(ws + p.off_stats),
                       (const float*)(ws + p.off_opart), (bf16_t*)out, lse, wsum,
                       chunk ? nullptr : scores_acc, (const int32_t*)nullptr);
}

hipError_t launch_decode_step_insert_first(const Shape& s, const Plan& p, const void* q,
                                           void* kc, void* vc, float* scores, int32_t* token_pos,
                                           const void* kn, const void* vn, void* out, float* lse,
                                           float* wsum, int32_t* evict_idx, int32_t pos0,
                                           char* ws, float scale, hipStream_t st) {
  const float c = scale * kLog2e;
  int ns = 0;
  hipError_t e = launch_decode_split(
      s, p, q, kc, vc, ws, c, KeyPos{token_pos, pos0}, st, &ns,
      InsArgs{scores, (const bf16_t*)kn, (const bf16_t*)vn, evict_idx});
  if (e != hipSuccess) return e;
  const dim3 cgrid((s.M + kCols - 1) / kCols, s.BH());
  auto combine = s.d == 64 ? decode_combine<64> : decode_combine<128>;
  return launch_kernel(K_DECODE_COMBINE, combine, cgrid, dim3(kCombThreads), st, (const bf16_t*)q,
                       (const bf16_t*)nullptr, (const bf16_t*)nullptr, s.Hq, s.Hkv, s.M, ns, c,
                       (const float*)(ws + p.off_logits), (const float2*)(ws + p.off_stats),
                       (const float*)(ws + p.off_opart), (bf16_t*)out, lse, wsum, scores,
                       (const int32_t*)evict_idx);
}

namespace {

// The finish kernel for this (d, G); out_too selects the fused form.
hipError_t launch_finish(const Shape& s, const Plan& p, bool out_too, int ns, const void* q,
                         void* kc, void* vc, const void* kn, const void* vn, void* out,
                         float* lse, float* wsum, float* scores, int32_t* token_pos,
                         int32_t* evict_idx, int32_t pos0, char* ws, float c, hipStream_t st) {
  const int G = s.G();
  auto go = [&](auto kern) {
    return launch_kernel(K_DECODE_FINISH, kern, dim3(s.BH()), dim3(kFinThreads), st,
                         (const bf16_t*)q, (bf16_t*)kc, (bf16_t*)vc, (const bf16_t*)kn,
                         (const bf16_t*)vn, s.Hq, s.Hkv, s.M, ns, c,
                         (const float*)(ws + p.off_logits), (const float2*)(ws + p.off_stats),
                         (const float*)(ws + p.off_opart), (bf16_t*)out, lse, wsum, scores,
                         token_pos, evict_idx, pos0);
  };
#define H2O_FIN(DD, GG) \
  return out_too ? go(decode_finish<DD, GG, true>) : go(decode_finish<DD, GG, false>)
  if (s.d == 64) {
    if (G == 1) H2O_FIN(64, 1);
    if (G == 2) H2O_FIN(64, 2);
    if (G == 4) H2O_FIN(64, 4);
    if (G == 8) H2O_FIN(64, 8);
  } else {
    if (G == 1) H2O_FIN(128, 1);
    if (G == 2) H2O_FIN(128, 2);
    if (G == 4) H2O_FIN(128, 4);
  }
#undef H2O_FIN
  return hipErrorInvalidValue;
}

// The split count the split kernel used for this shape (chunk mode).
int split_count_for(const Shape& s) {
  const int G = s.G();
  if (s.M == 0) return 0;
  if (s.d == 64) {
    if (G == 1) return split_count<64, 1, false>(s.M, s.BH());
    if (G == 2) return split_count<64, 2, false>(s.M, s.BH());
    if (G == 4) return split_count<64, 4, false>(s.M, s.BH());
    if (G == 8) return split_count<64, 8, false>(s.M, s.BH());
  } else {
    if (G == 1) return split_count<128, 1, false>(s.M, s.BH());
    if (G == 2) return split_count<128, 2, false>(s.M, s.BH());
    if (G == 4) return split_count<128, 4, false>(s.M, s.BH());
  }
  return 0;
}

}  // namespace

hipError_t launch_decode_attend(const Shape& s, const Plan& p, const void* q, const void* kc,
                                const void* vc, const void* kn, const void* vn, void* out,
                                float* lse, char* ws, float scale, hipStream_t st) {
  const float c = scale * kLog2e;
  int ns = 0;
  hipError_t e = launch_decode_split(s, p, q, kc, vc, ws, c, KeyPos{nullptr, 0}, st, &ns);
  if (e != hipSuccess) return e;
  auto combine = s.d == 64 ? decode_combine<64> : decode_combine<128>;
  return launch_kernel(K_DECODE_COMBINE, combine, dim3(1, s.BH()), dim3(kCombThreads), st,
                       (const bf16_t*)q, (const bf16_t*)kn, (const bf16_t*)vn, s.Hq, s.Hkv,
                       s.M, ns, c, (const float*)(ws + p.off_logits),
                       (const float2*)(ws + p.off_stats), (const float*)(ws + p.off_opart),
                       (bf16_t*)out, lse, (float*)nullptr, (float*)nullptr,
                       (const int32_t*)nullptr);
}

hipError_t launch_decode_evict(const Shape& s, const Plan& p, const void* q, void* kc, void* vc,
                               const void* kn, const void* vn, float* wsum, float* scores,
                               int32_t* token_pos, int32_t* evict_idx, int32_t pos0, char* ws,
                               float scale, hipStream_t st) {
  return launch_finish(s, p, false, split_count_for(s), q, kc, vc, kn, vn, nullptr, nullptr,
                       wsum, scores, token_pos, evict_idx, pos0, ws, scale * kLog2e, st);
}

hipError_t launch_decode_step(const Shape& s, const Plan& p, const void* q, void* kc, void* vc,
                              const void* kn, const void* vn, void* out, float* lse,
                              float* wsum, float* scores, int32_t* token_pos, int32_t* evict_idx,
                              int32_t pos0, char* ws, float scale, hipStream_t st) {
  const float c = scale * kLog2e;
  int ns = 0;
  hipError_t e = launch_decode_split(s, p, q, kc, vc, ws, c, KeyPos{nullptr, 0}, st, &ns);
  if (e != hipSuccess) return e;
  return launch_finish(s, p, true, ns, q, kc, vc, kn, vn, out, lse, wsum, scores, token_pos,
                       evict_idx, pos0, ws, c, st);
}

}  // namespace h2o
