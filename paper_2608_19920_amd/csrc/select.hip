// Column-sum reduce, H2O score accumulation, bottom-k selection and insert.
#include "internal.h"

namespace h2o {
namespace {

// ------------------------------------------------------------ colsum reduce
// wsum[bh][j] = sum over the partial slots p (in increasing p, so the result
// is bitwise reproducible) whose rows can see column j. With scores
// non-null, a chunk step's accumulation in the same pass: scores[bh][j] +=
// wsum[bh][j] for j < M, one float32 addition of the stored value (the bits
// of the separate accumulate kernel); with copy non-null the sum is also
// written to copy[bh][j], the ranking input of the fused selection.
__global__ __launch_bounds__(256) void colsum_reduce_kernel(const float* __restrict__ parts,
                                                            float* __restrict__ wsum,
                                                            float* __restrict__ scores,
                                                            float* __restrict__ copy, int nparts,
                                                            int rows_per_part, int BH, int Nk,
                                                            int ld, int G, int T, int M,
                                                            int Tk) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  const int bh = blockIdx.y;
  if (j >= Nk) return;
  // the score is requested with the partials, not after them
  float* sc = scores && j < M ? scores + (size_t)bh * M + j : nullptr;
  const float s_old = sc ? *sc : 0.f;
  // The partials that see column j are p0 .. nparts-1 (kv_end grows with
  // p): all of them for a cache column, and for chunk key i = j - M those
  // whose last row (r1 - 1) / G reaches i, i.e. (p + 1) * rows_per_part > i * G.
  int p0 = 0;
  if (Tk > 0 && j >= M) p0 = ((j - M) * G) / rows_per_part;
  const float* src = parts + ((size_t)p0 * BH + bh) * ld + j;
  const size_t stride = (size_t)BH * ld;
  float s = 0.f;
  int p = p0;
  // sixteen loads in flight, additions in increasing p (bitwise reproducible)
  for (; p + 15 < nparts; p += 16, src += 16 * stride) {
    float a[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) a[e] = src[e * stride];
#pragma unroll
    for (int e = 0; e < 16; ++e) s += a[e];
  }
  for (; p + 3 < nparts; p += 4, src += 4 * stride) {
    const float a0 = src[0], a1 = src[stride], a2 = src[2 * stride], a3 = src[3 * stride];
    s += a0;
    s += a1;
    s += a2;
    s += a3;
  }
  for (; p < nparts; ++p, src += stride) s += src[0];
  wsum[(size_t)bh * Nk + j] = s;
  if (sc) {
    const float acc = s_old + s;
    *sc = acc;
    if (copy) copy[(size_t)bh * M + j] = acc;
  }
}

// ---------------------------------------------------------------- accumulate
__global__ __launch_bounds__(256) void accumulate_kernel(float* __restrict__ scores,
                                                         const float* __restrict__ wsum, int M,
                                                         int T) {
  const int row = blockIdx.y;
  const float* w = wsum + (size_t)row * (M + T);
  float* s = scores + (size_t)row * M;
  for (int j = blockIdx.x * blockDim.x + threadIdx.x; j < M; j += gridDim.x * blockDim.x)
    s[j] = s[j] + w[j];
}

// ------------------------------------------------------------------ bottom-k

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;

__device__ __forceinline__ uint32_t umin(uint32_t a, uint32_t b) { return a < b ? a : b; }

// Inclusive prefix sum over the 64 lanes of a wave with DPP moves: shifts by
// 1, 2, 4 and 8 lanes inside each 16-lane row (lanes shifted in from outside
// the row add 0), then the running total carried across rows by the
// broadcasts of lane 15 (into rows 1 and 3) and of lane 31 (into rows 2 and
// 3). Six VALU additions, no LDS permutes.
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x) {
  constexpr bool kZero = true;   // out-of-row source lanes read 0
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, kZero);   // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, kZero);   // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, kZero);   // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, kZero);   // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false);   // row_bcast:15
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xC, 0xF, false);   // row_bcast:31
  return x;
}

// Exclusive prefix sum over the block (thread order); also returns the total.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* tmp,
                                                         uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t x = wave_inclusive_scan(v);
  if (lane == 63) tmp[wave] = x;
  __syncthreads();
  if (wave == 0) {
    const uint32_t w = lane < kSelWaves ? tmp[lane] : 0u;
    const uint32_t z = wave_inclusive_scan(w);
    if (lane < kSelWaves) tmp[kSelWaves + lane] = z - w;   // exclusive wave offsets
    if (lane == kSelWaves - 1) tmp[2 * kSelWaves] = z;
  }
  __syncthreads();
  const uint32_t res = tmp[kSelWaves + wave] + x - v;
  *total = tmp[2 * kSelWaves];
  __syncthreads();
  return res;
}

// Rows of at most this many slots are staged in LDS as order keys (one pad
// word after every 32, so that a thread's contiguous chunk in the compaction
// and the strided reads of the histogram passes are both free of bank
// conflicts); longer rows are read from global memory in every pass.
constexpr int kSelLdsMax = 32768;
__device__ __forceinline__ int sel_lds_index(int j) { return j + (j >> 5); }

// hist[bin] += 1 for every active lane: plain LDS atomics. With 12-bit
// digits the keys of a row spread over many bins; measured on score rows,
// aggregating the lanes of a wave that share a bin (ballots, readlane) cost
// more than the conflicts it saves. A row of equal scores puts every lane of
// a wave on one bin, which serialises those atomics but stays correct.
__device__ __forceinline__ void hist_add(uint32_t* hist, uint32_t bin, bool active) {
  if (active) atomicAdd(&hist[bin], 1u);
}

// Radix digits of the 32-bit order key, most significant first.
constexpr int kSelBins = 4096;
constexpr int kSelShift[3] = {20, 8, 0};
constexpr uint32_t kSelDigitMask[3] = {0xFFFu, 0xFFFu, 0xFFu};
// A round of the block covers 4 consecutive slots per thread.
constexpr int kSelRound = 4 * kSelThreads;
constexpr int kSelChunkRounds = kSelLdsMax / kSelRound;   // rounds whose loads go out together

// Given the histogram of the current digit, the bin that holds the krem-th
// smallest key of the prefix, and the keys of the prefix below that bin:
// every thread sums four consecutive bins (and clears them for the next
// digit: only it reads them), a block scan gives each thread the count
// before its bins, and the one thread whose range holds the krem-th key
// writes the extended prefix, the rest of krem and the bin's count. Ends
// synced.
__device__ __forceinline__ void select_bin(uint32_t* hist, uint32_t* tmp, int shift,
                                           uint32_t prefix, uint32_t krem, uint32_t* sh_prefix,
                                           uint32_t* sh_krem, uint32_t* sh_count) {
  const int t = threadIdx.x;
  const uint32_t c0 = hist[4 * t], c1 = hist[4 * t + 1], c2 = hist[4 * t + 2],
                 c3 = hist[4 * t + 3];
  hist[4 * t] = hist[4 * t + 1] = hist[4 * t + 2] = hist[4 * t + 3] = 0u;
  const uint32_t c = c0 + c1 + c2 + c3;
  uint32_t total;
  const uint32_t before = block_exclusive_scan(c, tmp, &total);
  if (before < krem && before + c >= krem) {
    uint32_t b = before, bin = 4u * t;
    uint32_t cb = c0;
    if (b + c0 < krem) { b += c0; ++bin; cb = c1;
      if (b + c1 < krem) { b += c1; ++bin; cb = c2;
        if (b + c2 < krem) { b += c2; ++bin; cb = c3; } } }
    *sh_prefix = prefix | (bin << shift);
    *sh_krem = krem - b;
    *sh_count = cb;
  }
  __syncthreads();
}

// The four scores of a thread in round r of a chunk: slots base + r *
// kSelRound + 4 * t .. + 3 (16-byte loads where the row allows; slots past
// the row read as +inf and are not used).
__device__ __forceinline__ float4 load4(const float* s, int M, int j) {
  if (j + 3 < M && ((reinterpret_cast<uintptr_t>(s + j) & 15u) == 0))
    return *reinterpret_cast<const float4*>(s + j);
  float4 v;
  v.x = j < M ? s[j] : INFINITY;
  v.y = j + 1 < M ? s[j + 1] : INFINITY;
  v.z = j + 2 < M ? s[j + 2] : INFINITY;
  v.w = j + 3 < M ? s[j + 3] : INFINITY;
  return v;
}

// Radix selection of one row by one block: the k-th smallest key tau
// (digits of 12, 12 and 8 bits, most significant first; the first digit's
// histogram is taken while the row is staged; when the first digit's bin
// holds few keys they are gathered and ranked against each other instead of
// the last two digits, and in long rows those digits are taken over the
// gathered keys), then the compaction scan. Rows of up to kSelLdsMax slots
// are staged in LDS; longer rows are read from global memory in every pass.
// Every loop over the row takes rounds of the whole block (uniform trip
// counts: the gather takes ballots) with 4 slots per thread, so a thread
// has 4 independent reads in flight.
//
// Compaction in slot order: thread t owns the contiguous chunk [t*C,
// (t+1)*C). The slots of a chunk below tau come first in it, and the keys
// equal to tau of lowest slot are taken first, so a thread writes at
//   (slots below tau in earlier chunks) + min(keys equal to tau in earlier
//   chunks, need_eq)
// - one block scan of both counts, packed in 16-bit halves when the row is
// shorter than 65536 slots. Chunks of at most 32 slots keep the slots below
// and equal to tau as bit masks, so the emit does not read the keys again.
struct SelChunk {
  uint32_t tau;       // the k-th smallest key
  uint32_t take_eq;   // keys equal to tau this chunk contributes
  uint32_t w;         // output position of the chunk's first chosen slot
  int j0, j1;         // the chunk
  bool masks;         // lt_mask / eq_mask hold the chunk's keys (C <= 32)
  uint32_t lt_mask, eq_mask;
};

// Keys of the first digit's chosen bin gathered into LDS, at most.
constexpr int kSelCand = 2048;
// Gathered keys ranked against each other instead of two more digits, at most.
constexpr int kSelRankMax = 256;

// sh_ncand[0] receives the count of the chosen bin, sh_ncand[1] is the
// gather's counter.
template <bool LDS>
__device__ __forceinline__ SelChunk bottomk_select(const float* s, int M, int k, uint32_t* keys,
                                                   uint32_t* hist, uint32_t* tmp, uint32_t* cand,
                                                   uint32_t* sh_ncand, uint32_t* sh_prefix,
                                                   uint32_t* sh_krem) {
  static_assert(kSelBins == 4 * kSelThreads, "four bins per thread in select_bin");
  const int t4 = 4 * (int)threadIdx.x;
  auto key_at = [&](int j) { return LDS ? keys[sel_lds_index(j)] : order_key(s[j]); };
  for (int b = threadIdx.x; b < kSelBins; b += kSelThreads) hist[b] = 0u;
  if (threadIdx.x == 0) sh_ncand[1] = 0u;   // the gather's counter
  __syncthreads();
  // first digit while the keys are staged: the loads of a chunk of rounds
  // (the whole row when it fits LDS) are issued before their keys are used
  for (int base = 0; base < M; base += kSelLdsMax) {
    float4 v[kSelChunkRounds];
#pragma unroll
    for (int r = 0; r < kSelChunkRounds; ++r)
      if (base + r * kSelRound < M) v[r] = load4(s, M, base + r * kSelRound + t4);
#pragma unroll
    for (int r = 0; r < kSelChunkRounds; ++r) {
      if (base + r * kSelRound >= M) break;   // uniform
      const float f[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = base + r * kSelRound + t4 + e;
        const uint32_t key = order_key(f[e]);
        if (LDS && j < M) keys[sel_lds_index(j)] = key;
        hist_add(hist, key >> kSelShift[0], j < M);
      }
    }
  }
  __syncthreads();
  select_bin(hist, tmp, kSelShift[0], 0u, (uint32_t)k, sh_prefix, sh_krem, sh_ncand);
  uint32_t prefix = *sh_prefix, krem = *sh_krem;
  uint32_t mask = kSelDigitMask[0] << kSelShift[0];
  // The keys of the chosen first-digit bin: when there are at most
  // kSelRankMax of them (the usual case, 12-bit digits spreading a row over
  // many bins), or in rows of 16,384 slots or more at most kSelCand, one
  // pass over the row gathers them into LDS. A few are ranked against each
  // other; more take the two remaining digits, histogrammed over the list
  // instead of over the row (in shorter rows two passes over the row cost
  // no more than the gather). Each wave reserves its lanes' places with one
  // atomic add.
  const uint32_t nb = *sh_ncand;   // keys in the chosen bin
  const bool rank = nb <= (uint32_t)kSelRankMax;                       // uniform
  const bool gather = rank || (M >= 16 * kSelThreads && nb <= (uint32_t)kSelCand);
  if (gather) {
    const int lane = threadIdx.x & 63;
    for (int j0 = 0; j0 < M; j0 += kSelRound) {
      uint32_t kk[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = j0 + t4 + e;
        kk[e] = j < M ? key_at(j) : 0u;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool in = j0 + t4 + e < M && (kk[e] & mask) == prefix;
        const uint64_t bal = __ballot(in);
        if (bal) {   // uniform over the wave
          uint32_t base = 0u;
          if (lane == 0) base = atomicAdd(sh_ncand + 1, (uint32_t)__popcll(bal));
          base = __builtin_amdgcn_readfirstlane(base);
          if (in) cand[base + (uint32_t)__popcll(bal & ((1ull << lane) - 1ull))] = kk[e];
        }
      }
    }
    __syncthreads();
  }
  if (rank) {
    // tau is the gathered value x with fewer than krem smaller keys and at
    // least krem keys <= x (the krem-th smallest of the bin); the threads
    // holding a key equal to it write the same values
    if (threadIdx.x < nb) {
      const uint32_t x = cand[threadIdx.x];
      uint32_t lt = 0u, le = 0u;
      const uint4* c4 = reinterpret_cast<const uint4*>(cand);
      const uint32_t nq = nb >> 2;
      for (uint32_t i = 0; i < nq; ++i) {
        const uint4 y = c4[i];
        lt += (uint32_t)(y.x < x) + (uint32_t)(y.y < x) + (uint32_t)(y.z < x) +
              (uint32_t)(y.w < x);
        le += (uint32_t)(y.x <= x) + (uint32_t)(y.y <= x) + (uint32_t)(y.z <= x) +
              (uint32_t)(y.w <= x);
      }
      for (uint32_t i = nq << 2; i < nb; ++i) {
        const uint32_t y = cand[i];
        lt += (uint32_t)(y < x);
        le += (uint32_t)(y <= x);
      }
      if (lt < krem && krem <= le) {
        *sh_prefix = x;
        *sh_krem = krem - lt;
      }
    }
    __syncthreads();
    prefix = *sh_prefix;
    krem = *sh_krem;
  }
#pragma unroll
  for (int d = 1; d < 3; ++d) {
    if (rank) break;   // uniform
    // (select_bin left the histogram cleared)
    if (gather) {
      for (int i = threadIdx.x; i < (int)nb; i += kSelThreads) {
        const uint32_t key = cand[i];
        hist_add(hist, (key >> kSelShift[d]) & kSelDigitMask[d], (key & mask) == prefix);
      }
    } else {
      for (int j0 = 0; j0 < M; j0 += kSelRound) {
        uint32_t kk[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = j0 + t4 + e;
          kk[e] = j < M ? key_at(j) : 0u;
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
          hist_add(hist, (kk[e] >> kSelShift[d]) & kSelDigitMask[d],
                   j0 + t4 + e < M && (kk[e] & mask) == prefix);
      }
    }
    __syncthreads();
    select_bin(hist, tmp, kSelShift[d], prefix, krem, sh_prefix, sh_krem, sh_ncand);
    prefix = *sh_prefix;
    krem = *sh_krem;
    mask |= kSelDigitMask[d] << kSelShift[d];
  }
  SelChunk c;
  c.tau = prefix;
  const uint32_t need_eq = krem;
  const int C = (M + kSelThreads - 1) / kSelThreads;
  c.j0 = min(M, (int)threadIdx.x * C);
  c.j1 = min(M, c.j0 + C);
  c.masks = C <= 32;
  uint32_t n_less = 0, n_eq = 0, lt_mask = 0, eq_mask = 0;
#pragma unroll 4
  for (int j = c.j0; j < c.j1; ++j) {
    const uint32_t key = key_at(j);
    const uint32_t bit = 1u << ((j - c.j0) & 31);
    if (key < c.tau) { ++n_less; lt_mask |= bit; }
    if (key == c.tau) { ++n_eq; eq_mask |= bit; }
  }
  c.lt_mask = lt_mask;
  c.eq_mask = eq_mask;
  uint32_t tot, less_before, eq_before;
  if (M < 65536) {
    const uint32_t both = block_exclusive_scan(n_less | (n_eq << 16), tmp, &tot);
    less_before = both & 0xFFFFu;
    eq_before = both >> 16;
  } else {
    less_before = block_exclusive_scan(n_less, tmp, &tot);
    eq_before = block_exclusive_scan(n_eq, tmp, &tot);
  }
  // keys equal to tau taken before this chunk, and by it (the difference
  // need_eq - eq_taken never wraps, so no guarded subtraction is needed: a
  // guarded one let the optimiser drop the cap below)
  const uint32_t eq_taken = umin(eq_before, need_eq);
  c.take_eq = umin(n_eq, need_eq - eq_taken);
  c.w = less_before + eq_taken;
  return c;
}

// Calls f(slot, position) for every chosen slot of the thread's chunk, in
// increasing slot order, with consecutive positions from c.w on (positions
// below k only).
template <bool LDS, typename F>
__device__ __forceinline__ void bottomk_emit(const SelChunk& c, const float* s,
                                             const uint32_t* keys, int k, F&& f) {
  uint32_t w = c.w;
  if (c.masks) {
    // the lowest take_eq bits of eq_mask
    uint32_t em = c.eq_mask, sel = c.lt_mask;
    for (uint32_t i = 0; i < c.take_eq; ++i) {
      const uint32_t low = em & (0u - em);
      sel |= low;
      em ^= low;
    }
    while (sel) {
      const int b = __ffs((int)sel) - 1;
      sel &= sel - 1;
      if (w < (uint32_t)k) f(c.j0 + b, w++);
    }
  } else {
    uint32_t eq_seen = 0;
    for (int j = c.j0; j < c.j1; ++j) {
      const uint32_t key = LDS ? keys[sel_lds_index(j)] : order_key(s[j]);
      bool sel = key < c.tau;
      if (key == c.tau) { sel = eq_seen < c.take_eq; ++eq_seen; }
      if (sel && w < (uint32_t)k) f(j, w++);
    }
  }
}

// One block per row: emit, in ascending slot order, every slot with key <
// tau and the lowest-index (k - #less) slots with key == tau.
template <bool LDS>
__global__ __launch_bounds__(kSelThreads) void bottomk_kernel(const float* __restrict__ scores,
                                                              int M, int k,
                                                              int32_t* __restrict__ idx) {
  __shared__ uint32_t keys[LDS ? kSelLdsMax + kSelLdsMax / 32 : 1];
  __shared__ uint32_t hist[kSelBins];
  __shared__ uint32_t tmp[2 * kSelWaves + 1];
  __shared__ __attribute__((aligned(16))) uint32_t cand[kSelCand];
  __shared__ uint32_t sh_ncand[2], sh_prefix, sh_krem;
  const float* s = scores + (size_t)blockIdx.x * M;
  int32_t* out = idx + (size_t)blockIdx.x * k;
  if (k <= 0) return;
  const SelChunk c =
      bottomk_select<LDS>(s, M, k, keys, hist, tmp, cand, sh_ncand, &sh_prefix, &sh_krem);
  bottomk_emit<LDS>(c, s, keys, k, [&](int j, uint32_t w) { out[w] = j; });
}

// Selection and insert in one launch. Block (row, x), x < X = gridDim.y,
// ranks the row's keys (which no kernel writes while it runs: a copy of the
// accumulated scores), every one of the X blocks of a row computing the same
// selection, so they need no communication. The X blocks of a row are
// dispatched `rows` slots apart, so with a row count that is a multiple of
// 8 they land on one XCD (dispatch goes round-robin over the 8) and read
// the row through one L2. The chunk of thread t is
// written out (evict_idx, the inserted slots' scores and token positions)
// by block t % X; block x copies the K/V rows of chunk tokens [x*k/X,
// (x+1)*k/X) into their slots, whose indices every block keeps in LDS (the
// histogram array, free after the selection; k <= kSelBins). Same results
// as bottomk_kernel followed by insert_kernel.
template <bool LDS>
__global__ __launch_bounds__(kSelThreads) void bottomk_insert_kernel(
    const float* __restrict__ keys_in, float* __restrict__ scores,
    int32_t* __restrict__ token_pos, uint4* __restrict__ kc, uint4* __restrict__ vc,
    const uint4* __restrict__ kn, const uint4* __restrict__ vn, const float* __restrict__ wsum,
    int32_t* __restrict__ idx, int M, int T, int k, int vecs, int32_t pos0) {
  __shared__ uint32_t keys[LDS ? kSelLdsMax + kSelLdsMax / 32 : 1];
  __shared__ uint32_t hist[kSelBins];
  __shared__ uint32_t tmp[2 * kSelWaves + 1];
  __shared__ __attribute__((aligned(16))) uint32_t cand[kSelCand];
  __shared__ uint32_t sh_ncand[2], sh_prefix, sh_krem;
  const size_t row = blockIdx.x;
  const int X = gridDim.y, x = blockIdx.y;
  const float* s = keys_in + row * M;
  if (k <= 0) return;
  const SelChunk c =
      bottomk_select<LDS>(s, M, k, keys, hist, tmp, cand, sh_ncand, &sh_prefix, &sh_krem);
  uint32_t* sidx = hist;   // k <= kSelBins
  const bool own = (int)threadIdx.x % X == x;
  bottomk_emit<LDS>(c, s, keys, k, [&](int j, uint32_t w) {
    sidx[w] = (uint32_t)j;
    if (own) {
      idx[row * k + w] = j;
      scores[row * M + j] = wsum ? wsum[row * (size_t)(M + T) + M + w] : 0.f;
      if (token_pos) token_pos[row * M + j] = pos0 + (int32_t)w;
    }
  });
  __syncthreads();
  // chunk tokens [i0, i1) of this block: 16-byte vectors, four loads of each
  // tensor in flight per thread before the stores
  const int i0 = (int)((long long)k * x / X), i1 = (int)((long long)k * (x + 1) / X);
  const int n = (i1 - i0) * vecs;
  constexpr int U = 4;
  for (int e0 = threadIdx.x; e0 < n; e0 += U * kSelThreads) {
    uint4 kv[U], vv[U];
    uint32_t slot[U];
    int cc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = e0 + u * kSelThreads;
      slot[u] = 0xFFFFFFFFu;
      cc[u] = 0;
      if (e < n) {
        const int i = i0 + e / vecs;
        cc[u] = e % vecs;
        kv[u] = kn[(row * T + i) * vecs + cc[u]];
        vv[u] = vn[(row * T + i) * vecs + cc[u]];
        slot[u] = sidx[i];
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (slot[u] < (uint32_t)M) {
        kc[(row * M + slot[u]) * vecs + cc[u]] = kv[u];
        vc[(row * M + slot[u]) * vecs + cc[u]] = vv[u];
      }
    }
  }
}

// -------------------------------------------------------------------- insert
// Block (x, row) copies chunk keys/values i in [x*kPer, x*kPer + kPer) into
// their evicted slots, 16 bytes per thread per step.
constexpr int kInsThreads = 256;

__global__ __launch_bounds__(kInsThreads) void insert_kernel(
    uint4* __restrict__ kc, uint4* __restrict__ vc, float* __restrict__ scores,
    int32_t* __restrict__ token_pos, const uint4* __restrict__ kn, const uint4* __restrict__ vn,
    const float* __restrict__ wsum, const int32_t* __restrict__ idx, int M, int T, int vecs,
    int k, int kPer, int32_t pos0) {
  const size_t row = blockIdx.y;
  const int i0 = blockIdx.x * kPer;
  const int n = min(kPer, k - i0);
  for (int e = threadIdx.x; e < n * vecs; e += kInsThreads) {
    const int i = i0 + e / vecs, c = e % vecs;
    const int slot = idx[row * k + i];
    if ((unsigned)slot >= (unsigned)M) continue;
    kc[(row * M + slot) * vecs + c] = kn[(row * T + i) * vecs + c];
    vc[(row * M + slot) * vecs + c] = vn[(row * T + i) * vecs + c];
  }
  for (int e = threadIdx.x; e < n; e += kInsThreads) {
    const int i = i0 + e;
    const int slot = idx[row * k + i];
    if ((unsigned)slot >= (unsigned)M) continue;
    scores[row * M + slot] = wsum ? wsum[row * (size_t)(M + T) + M + i] : 0.f;
    if (token_pos) token_pos[row * M + slot] = pos0 + i;
  }
}

// k == 1 (token generation): the (score, slot)-smallest slot of each row and
// the insert into it, one block per row.
constexpr int kArgThreads = 256;

// The ranked values come from `keys` (the scores themselves, or a score
// variant), row `row` or, with key_rows > 0, row `row % key_rows` (one key
// row shared by the batch).
__global__ __launch_bounds__(kArgThreads) void argmin_insert_kernel(
    uint4* __restrict__ kc, uint4* __restrict__ vc, float* scores, const float* keys,
    int key_rows, int32_t* __restrict__ token_pos, const uint4* __restrict__ kn,
    const uint4* __restrict__ vn, const float* __restrict__ wsum, int32_t* __restrict__ idx,
    int M, int T, int vecs, int32_t pos0) {
  __shared__ uint32_t red_hi[kArgThreads / 64], red_lo[kArgThreads / 64];
  __shared__ int sh_slot;
  const size_t row = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* s = keys + (key_rows > 0 ? row % key_rows : row) * M;
  // (key, slot), lexicographic; the start (max key, slot 0) is a real pair
  // whenever every key is the maximum, so the result is always a slot
  uint32_t bk = 0xFFFFFFFFu, bj = 0u;
  // four independent loads per step; slots are visited in increasing order
  // per thread, so a strict < keeps the lowest slot among equal keys
  int j = tid;
  for (; j + 3 * kArgThreads < M; j += 4 * kArgThreads) {
    float v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = s[j + u * kArgThreads];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint32_t key = order_key(v[u]);
      if (key < bk) { bk = key; bj = (uint32_t)(j + u * kArgThreads); }
    }
  }
  for (; j < M; j += kArgThreads) {
    const uint32_t key = order_key(s[j]);
    if (key < bk) { bk = key; bj = (uint32_t)j; }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t ok = __shfl_xor(bk, o, 64), oj = __shfl_xor(bj, o, 64);
    if (ok < bk || (ok == bk && oj < bj)) { bk = ok; bj = oj; }
  }
  if (lane == 0) { red_hi[wave] = bk; red_lo[wave] = bj; }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < kArgThreads / 64; ++w)
      if (red_hi[w] < bk || (red_hi[w] == bk && red_lo[w] < bj)) { bk = red_hi[w]; bj = red_lo[w]; }
    const int slot = (int)bj;
    sh_slot = slot;
    idx[row] = slot;
    if ((unsigned)slot < (unsigned)M) {
      scores[row * M + slot] = wsum ? wsum[row * (size_t)(M + T) + M] : 0.f;
      if (token_pos) token_pos[row * M + slot] = pos0;
    }
  }
  __syncthreads();
  const int slot = sh_slot;
  if ((unsigned)slot >= (unsigned)M) return;
  for (int c = tid; c < vecs; c += kArgThreads) {
    kc[(row * M + slot) * vecs + c] = kn[(row * T) * vecs + c];
    vc[(row * M + slot) * vecs + c] = vn[(row * T) * vecs + c];
  }
}

}  // namespace

hipError_t launch_argmin_insert(void* kc, void* vc, float* scores, const float* keys,
                                int key_rows, int32_t* token_pos, const void* kn, const void* vn,
                                const float* wsum, int32_t* idx, int rows, int M, int T, int d,
                                int32_t pos0, int elem_bytes, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  return launch_kernel(K_ARGMIN_INSERT, argmin_insert_kernel, dim3(rows), dim3(kArgThreads), st,
                       (uint4*)kc, (uint4*)vc, scores, keys, key_rows, token_pos,
                       (const uint4*)kn, (const uint4*)vn, wsum, idx, M, T,
                       d * elem_bytes / 16, pos0);
}

// ------------------------------------------------------- score variants
// h2o_norm: keys = scores / (t - token_pos), one correctly rounded float32
// division per slot (the age is exact in float32 below 2^24). n = rows * M.
__global__ __launch_bounds__(256) void norm_keys_kernel(const float* __restrict__ scores,
                                                        const int32_t* __restrict__ token_pos,
                                                        float* __restrict__ keys, size_t n,
                                                        int32_t t) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    keys[i] = scores[i] / (float)(t - token_pos[i]);
}

// h2o_orig: keys[h, j] = sum over b of scores[b, h, j], float32 additions in
// increasing b. n = Hkv * M, the size of one batch entry's scores.
__global__ __launch_bounds__(256) void orig_keys_kernel(const float* __restrict__ scores,
                                                        float* __restrict__ keys, int B,
                                                        size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x) {
    float a = scores[i];
    for (int b = 1; b < B; ++b) a += scores[(size_t)b * n + i];
    keys[i] = a;
  }
}

// dst[b, :] = src[:] for every b (n = Hkv * k indices per batch entry).
__global__ __launch_bounds__(256) void broadcast_rows_kernel(const int32_t* __restrict__ src,
                                                             int32_t* __restrict__ dst, int B,
                                                             size_t n) {
  const size_t total = (size_t)B * n;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (size_t)gridDim.x * blockDim.x)
    dst[i] = src[i % n];
}

namespace {
// Grid of an elementwise pass over n items: 256 threads, at most 4096 blocks
// (16 per CU), grid-stride beyond that.
unsigned flat_blocks(size_t n) {
  const size_t b = (n + 255) / 256;
  return (unsigned)(b < 4096 ? b : 4096);
}
}  // namespace

hipError_t launch_norm_keys(const float* scores, const int32_t* token_pos, float* keys, int rows,
                            int M, int32_t t, hipStream_t st) {
  const size_t n = (size_t)rows * M;
  if (n == 0) return hipSuccess;
  return launch_kernel(K_KEYS, norm_keys_kernel, dim3(flat_blocks(n)), dim3(256), st, scores,
                       token_pos, keys, n, t);
}

hipError_t launch_orig_keys(const float* scores, float* keys, int B, int Hkv, int M,
                            hipStream_t st) {
  const size_t n = (size_t)Hkv * M;
  if (n == 0) return hipSuccess;
  return launch_kernel(K_KEYS, orig_keys_kernel, dim3(flat_blocks(n)), dim3(256), st, scores,
                       keys, B, n);
}

hipError_t launch_broadcast_rows(const int32_t* src, int32_t* dst, int B, int n,
                                 hipStream_t st) {
  const size_t total = (size_t)B * n;
  if (total == 0) return hipSuccess;
  return launch_kernel(K_KEYS, broadcast_rows_kernel, dim3(flat_blocks(total)), dim3(256), st,
                       src, dst, B, (size_t)n);
}

hipError_t launch_colsum_reduce(const Shape& s, const Plan& p, const float* parts, float* wsum,
                                hipStream_t st, ScoreAcc acc) {
  dim3 grid((s.Nk() + 255) / 256, s.BH());
  return launch_kernel(K_COLSUM_REDUCE, colsum_reduce_kernel, grid, dim3(256), st, parts, wsum,
                       acc.scores, acc.scores ? acc.copy : nullptr, p.nparts, p.rows_per_part,
                       s.BH(), s.Nk(), p.parts_ld, s.G(), s.T, s.M, s.Tk());
}

hipError_t launch_accumulate(float* scores, const float* wsum, int rows, int M, int T,
                             hipStream_t st) {
  if (rows == 0 || M == 0) return hipSuccess;
  int bx = (M + 256 * 4 - 1) / (256 * 4);
  dim3 grid(bx < 1 ? 1 : bx, rows);
  return launch_kernel(K_ACCUMULATE, accumulate_kernel, grid, dim3(256), st, scores, wsum, M, T);
}

hipError_t launch_bottomk(const float* scores, int rows, int M, int k, int32_t* idx,
                          hipStream_t st) {
  if (rows == 0 || k == 0) return hipSuccess;
  if (M <= kSelLdsMax)
    return launch_kernel(K_BOTTOMK, bottomk_kernel<true>, dim3(rows), dim3(kSelThreads), st,
                         scores, M, k, idx);
  return launch_kernel(K_BOTTOMK, bottomk_kernel<false>, dim3(rows), dim3(kSelThreads), st,
                       scores, M, k, idx);
}

bool bottomk_insert_supported(int k) { return k >= 1 && k <= kSelBins; }

hipError_t launch_bottomk_insert(const float* keys, float* scores, int32_t* token_pos, void* kc,
                                 void* vc, const void* kn, const void* vn, const float* wsum,
                                 int32_t* idx, int rows, int M, int T, int d, int k,
                                 int32_t pos0, int elem_bytes, hipStream_t st) {
  if (rows == 0 || k == 0) return hipSuccess;
  if (!bottomk_insert_supported(k)) return hipErrorInvalidValue;
  // about one block per CU in all: the X blocks of a row repeat its
  // selection and share its inserts (8 to 32 blocks per row measured: the
  // copy, not the repeated selection, decides)
  int X = 256 / rows;
  if (X > 32) X = 32;
  if (X < 1) X = 1;
  const int vecs = d * elem_bytes / 16;
  const dim3 grid(rows, X);
  if (M <= kSelLdsMax)
    return launch_kernel(K_BOTTOMK_INSERT, bottomk_insert_kernel<true>, grid, dim3(kSelThreads), st,
                         keys, scores, token_pos, (uint4*)kc, (uint4*)vc, (const uint4*)kn,
                         (const uint4*)vn, wsum, idx, M, T, k, vecs, pos0);
  return launch_kernel(K_BOTTOMK_INSERT, bottomk_insert_kernel<false>, grid, dim3(kSelThreads), st,
                       keys, scores, token_pos, (uint4*)kc, (uint4*)vc, (const uint4*)kn,
                       (const uint4*)vn, wsum, idx, M, T, k, vecs, pos0);
}

hipError_t launch_insert(void* kc, void* vc, float* scores, int32_t* token_pos, const void* kn,
                         const void* vn, const float* wsum, const int32_t* idx, int rows, int M,
                         int T, int d, int k, int32_t pos0, int elem_bytes, hipStream_t st) {
  if (rows == 0 || k == 0) return hipSuccess;
  const int vecs = d * elem_bytes / 16;
  int kPer = kInsThreads / vecs;
  if (kPer < 1) kPer = 1;
  dim3 grid((k + kPer - 1) / kPer, rows);
  return launch_kernel(K_INSERT, insert_kernel, grid, dim3(kInsThreads), st, (uint4*)kc,
                       (uint4*)vc, scores, token_pos, (const uint4*)kn, (const uint4*)vn, wsum,
                       idx, M, T, vecs, k, kPer, pos0);
}

}  // namespace h2o
