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
#include "internal.h"

namespace h2o {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kStep = 32;                                // cache slots per wave step
constexpr int kMaxGD = 512;                              // G * D handled by these kernels
constexpr int kMaxSplit = 64;                            // split blocks per head, at most
constexpr int kBufferFlags = 0x00020000;                 // buffer descriptor word 3 (32-bit data)

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
template <int D, int G>
__global__ __launch_bounds__(kThreads) void decode_split(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    int Hq, int Hkv, int M, float c_log2, float* __restrict__ logits,
    float2* __restrict__ dstat, float* __restrict__ dO, float* __restrict__ sink) {
  constexpr int DH = D / 32;                 // MFMA k-chunks of a row
  constexpr int NK = 2 * DH;                 // K loads per step (two 16-slot blocks)
  constexpr int RPL = 512 / D;               // V rows per wave load
  constexpr int NV = kStep / RPL;            // V loads per step
  constexpr int VP = vpitch<D>();
  static_assert(G <= 16 && (D == 64 || D == 128), "decode shape");
  __shared__ __attribute__((aligned(16))) bf16_t vs_all[kWaves][kStep * VP];
  __shared__ float red_m[kWaves][16], red_l[kWaves][16];
  __shared__ float ored[kWaves][G][D];
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
  const int head_bytes = (int)((uint32_t)M * (uint32_t)(D * 2));
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(kc + bh * (size_t)M * D), (short)0, head_bytes, kBufferFlags);
  const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(vc + bh * (size_t)M * D), (short)0, head_bytes, kBufferFlags);
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
  auto issue = [&](int k, int u) {
    const uint32_t base = (uint32_t)((stream + k * nstreams) * kStep) * (uint32_t)(D * 2);
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

  auto consume = [&](int k, int u) {
    const int key0 = (stream + k * nstreams) * kStep;
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
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      lg[i] = sacc[i >> 2][i & 3] * c_log2;
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
      const float p = key < M ? __builtin_amdgcn_exp2f(lg[i] - m) : 0.f;
      l += p;
      pb[i] = (__bf16)p;
    }
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int db = 0; db < D / 16; ++db) oacc[db] = mfma(v_operand<D>(vs, db, lane), pb, oacc[db]);
  };

  issue(0, 0);
  for (int k = 0; k < nst; k += 2) {
    issue(k + 1, 1);
    consume(k, 0);
    if (k + 1 >= nst) break;
    issue(k + 2, 0);
    consume(k + 1, 1);
  }
  // block merge: per column, the common maximum over the waves
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  if (grp == 0) {
    red_m[wave][col] = m;
    red_l[wave][col] = l;
  }
  __syncthreads();
  float mb = red_m[0][col];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) mb = fmaxf(mb, red_m[w][col]);
  const float sc = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - mb);
  if (col < G) {
#pragma unroll
    for (int db = 0; db < D / 16; ++db)
#pragma unroll
      for (int r = 0; r < 4; ++r) ored[wave][col][16 * db + 4 * grp + r] = oacc[db][r] * sc;
  }
  __syncthreads();
  if (tid < G) {
    float mg = red_m[0][tid];
    for (int w = 1; w < kWaves; ++w) mg = fmaxf(mg, red_m[w][tid]);
    float lt = 0.f;
    for (int w = 0; w < kWaves; ++w)
      if (red_m[w][tid] != -INFINITY) lt += red_l[w][tid] * __builtin_amdgcn_exp2f(red_m[w][tid] - mg);
    dstat[(bh * nsplit + s) * G + tid] = make_float2(mg, lt);
  }
  for (int c = tid; c < G * D; c += kThreads) {
    float a = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) a += ored[w][c / D][c % D];
    dO[(bh * nsplit + s) * (size_t)(G * D) + c] = a;
  }
}

// Block (x, bh): merges the splits of head bh (every block recomputes the
// few per-head statistics from the split partials staged in LDS), then
// writes wsum for columns [x*kCols, +kCols); block x == 0 also writes out
// and lse.
constexpr int kCols = 1024;

template <int D>
__global__ __launch_bounds__(kThreads) void decode_combine(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ kn, const bf16_t* __restrict__ vn,
    int Hq, int Hkv, int M, int nsplit, float c_log2, const float* __restrict__ logits,
    const float2* __restrict__ dstat, const float* __restrict__ dO, bf16_t* __restrict__ out,
    float* __restrict__ lse, float* __restrict__ wsum) {
  constexpr int kMaxG = kMaxGD / 64;
  __shared__ float lnew[kMaxG], lam[kMaxG], mfin[kMaxG], linv[kMaxG];
  __shared__ float2 st_s[kMaxSplit * kMaxG];
  const int G = Hq / Hkv;
  const size_t bh = blockIdx.y;
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < nsplit * G; i += kThreads) st_s[i] = dstat[bh * nsplit * G + i];
  // logit of the chunk's own key for each query head (one wave per head)
  for (int g = wave; g < G; g += kThreads / 64) {
    float a = 0.f;
    for (int dd = lane; dd < D; dd += 64)
      a = fmaf(bf16_to_f32(q[(size_t)(b * Hq + h * G + g) * D + dd]),
               bf16_to_f32(kn[bh * D + dd]), a);
    for (int o = 32; o > 0; o >>= 1) a += __shfl_xor(a, o, 64);
    if (lane == 0) lnew[g] = a * c_log2;
  }
  __syncthreads();
  if (tid < G) {
    const int g = tid;
    float mx = lnew[g];
    for (int s = 0; s < nsplit; ++s) mx = fmaxf(mx, st_s[s * G + g].x);
    float L = __builtin_amdgcn_exp2f(lnew[g] - mx);
    for (int s = 0; s < nsplit; ++s) {
      const float2 st = st_s[s * G + g];
      if (st.y > 0.f) L += st.y * __builtin_amdgcn_exp2f(st.x - mx);
    }
    const float lm = mx + __log2f(L);
    lam[g] = lm;
    mfin[g] = mx;
    linv[g] = 1.f / L;
    if (blockIdx.x == 0) lse[(size_t)(b * Hq + h * G + g)] = lm * kLn2;
  }
  __syncthreads();
  if (blockIdx.x == 0) {
    for (int c = tid; c < G * D; c += kThreads) {
      const int g = c / D, dd = c % D;
      float a = __builtin_amdgcn_exp2f(lnew[g] - mfin[g]) * bf16_to_f32(vn[bh * D + dd]);
#pragma unroll 8
      for (int s = 0; s < nsplit; ++s) {
        const float2 st = st_s[s * G + g];
        const float w = st.y > 0.f ? __builtin_amdgcn_exp2f(st.x - mfin[g]) : 0.f;
        a = fmaf(dO[(bh * nsplit + s) * (size_t)(G * D) + c], w, a);
      }
      out[(size_t)(b * Hq + h * G + g) * D + dd] = f32_to_bf16(a * linv[g]);
    }
  }
  float* w = wsum + bh * (size_t)(M + 1);
  const float* lgb = logits + bh * (size_t)G * logit_pitch(M);
  const int c0 = blockIdx.x * kCols, c1 = min(M, c0 + kCols);
  for (int j = c0 + tid; j < c1; j += kThreads) {
    float a = 0.f;
    for (int g = 0; g < G; ++g)
      a += __builtin_amdgcn_exp2f(lgb[(size_t)g * logit_pitch(M) + j] - lam[g]);
    w[j] = a;
  }
  if (blockIdx.x == 0 && tid == 0) {
    float a = 0.f;
    for (int g = 0; g < G; ++g) a += __builtin_amdgcn_exp2f(lnew[g] - lam[g]);
    w[M] = a;
  }
}

// Split blocks per head such that all blocks of the grid are resident at
// once (blocks per CU of this kernel instance x CUs), at most kMaxSplit and
// at most one wave per step of slots.
template <int D, int G>
int split_count(int M, int BH) {
  static int resident = 0;
  if (!resident) {
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, decode_split<D, G>, kThreads,
                                                     0) != hipSuccess || per_cu < 1)
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

template <int D, int G>
hipError_t launch_split(hipStream_t st, int BH, const void* q, const void* kc, const void* vc,
                        int Hq, int Hkv, int M, float c, float* logits, float2* dstat, float* dO,
                        float* sink, int* ns) {
  *ns = split_count<D, G>(M, BH);
  return launch_kernel(K_DECODE_SPLIT, decode_split<D, G>, dim3(*ns, BH), dim3(kThreads), st,
                       (const bf16_t*)q, (const bf16_t*)kc, (const bf16_t*)vc, Hq, Hkv, M, c,
                       logits, dstat, dO, sink);
}

}  // namespace

int decode_max_split() { return kMaxSplit; }

// The decode kernels are instantiated for these (d, G) pairs.
bool decode_supports(int d, int G) {
  return (d == 64 && (G == 1 || G == 2 || G == 4 || G == 8)) ||
         (d == 128 && (G == 1 || G == 2 || G == 4));
}

hipError_t launch_sdpa_decode(const Shape& s, const Plan& p, const void* q, const void* kc,
                              const void* vc, const void* kn, const void* vn, void* out,
                              float* lse, float* wsum, char* ws, float scale, hipStream_t st) {
  const float c = scale * kLog2e;
  float* logits = reinterpret_cast<float*>(ws + p.off_logits);
  float2* dstat = reinterpret_cast<float2*>(ws + p.off_stats);
  float* dO = reinterpret_cast<float*>(ws + p.off_opart);
  float* sink = reinterpret_cast<float*>(ws + p.off_parts);
  int ns = 0;
  if (s.M > 0) {
    const int G = s.G();
    hipError_t e = hipErrorInvalidValue;
#define H2O_SPLIT(DD, GG) \
  e = launch_split<DD, GG>(st, s.BH(), q, kc, vc, s.Hq, s.Hkv, s.M, c, logits, dstat, dO, sink, \
                           &ns)
    if (s.d == 64) {
      if (G == 1) H2O_SPLIT(64, 1);
      else if (G == 2) H2O_SPLIT(64, 2);
      else if (G == 4) H2O_SPLIT(64, 4);
      else if (G == 8) H2O_SPLIT(64, 8);
      else return hipErrorInvalidValue;
    } else {
      if (G == 1) H2O_SPLIT(128, 1);
      else if (G == 2) H2O_SPLIT(128, 2);
      else if (G == 4) H2O_SPLIT(128, 4);
      else return hipErrorInvalidValue;
    }
#undef H2O_SPLIT
    if (e != hipSuccess) return e;
  }
  const dim3 cgrid(s.M > 0 ? (s.M + kCols - 1) / kCols : 1, s.BH());
  auto combine = s.d == 64 ? decode_combine<64> : decode_combine<128>;
  return launch_kernel(K_DECODE_COMBINE, combine, cgrid, dim3(kThreads), st, (const bf16_t*)q,
                       (const bf16_t*)kn, (const bf16_t*)vn, s.Hq, s.Hkv, s.M, ns, c,
                       (const float*)logits, (const float2*)dstat, (const float*)dO,
                       (bf16_t*)out, lse, wsum);
}

}  // namespace h2o
