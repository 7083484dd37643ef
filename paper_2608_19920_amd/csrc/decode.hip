// Token generation (T = 1): the chunk is one query per query head, so the
// step streams the whole KV cache once and is bound by HBM bandwidth
// (Sec. "Sparse Attention. Key-Value Caching": N_q = 1, N_k = N_C).
//
//   split    block (split s, head bh) streams rounds s, s+ns, ... of head bh.
//            Sixteen lanes share one key row: lane `slice` holds D/16 elements
//            of it, so each wave load reads four consecutive rows (contiguous
//            bytes). Logits (log2 domain) reduce over the 16 lanes with DPP;
//            the split's softmax partial (m, l, O-partial) per query head is
//            written out, and so are the logits for the column sums.
//   combine  block bh merges the splits with the chunk's own key (column M),
//            writes out and lse, and wsum[j] = sum_g exp2(logit_gj - lambda_g)
//            from the stored logits.
#include "internal.h"

namespace h2o {
namespace {

constexpr int kThreads = 256;
constexpr int kLanesPerKey = 16;                         // lanes sharing one key row
constexpr int kKeysPerRound = kThreads / kLanesPerKey;   // 16
constexpr int kMaxGD = 512;                              // G * D handled by these kernels
constexpr int kMaxSplit = 64;                            // split blocks per head, at most

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, true));
}
// Sum over the 16 lanes of a DPP row; every lane gets the total.
__device__ __forceinline__ float sum16(float v) {
  v += dpp<0xB1>(v);    // quad_perm [1,0,3,2]
  v += dpp<0x4E>(v);    // quad_perm [2,3,0,1]
  v += dpp<0x141>(v);   // row_half_mirror: lane l <-> 7-l within each half row
  v += dpp<0x140>(v);   // row_mirror: lane l <-> 15-l
  return v;
}

// EPL consecutive bf16 elements of a row, as float.
template <int EPL>
struct RowPiece {
  typedef uint32_t raw_t __attribute__((ext_vector_type(EPL / 2)));
  static __device__ __forceinline__ raw_t load(const bf16_t* p) {
    return *reinterpret_cast<const raw_t*>(p);
  }
  static __device__ __forceinline__ void unpack(const raw_t w, float* f) {
#pragma unroll
    for (int e = 0; e < EPL / 2; ++e) {
      f[2 * e] = __uint_as_float(w[e] << 16);
      f[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
    }
  }
};

// Streaming split kernel. The cache slots of head bh are walked in rounds of
// 16 slots (one slot per 16-lane DPP row; lane `slice` holds D/16 elements
// of the row); block (s, bh) takes rounds s, s + ns, s + 2 ns, ... so that
// the ns blocks of a head sweep its K and V rows together. The K and V rows
// of the next PF rounds of a block are in flight while a round is computed.
// Each lane row keeps, per query head, a reference maximum m (the first
// logit it saw, raised only when a later logit exceeds it by more than 64 in
// log2 units, which keeps every exp2 term below 2^64), the sum l of
// exp2(logit - m) and the weighted V accumulator; the block merges them at
// the end.
template <int D, int G, int PF>
__global__ __launch_bounds__(kThreads) void decode_split(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    int Hq, int Hkv, int M, float c_log2, float* __restrict__ logits,
    float2* __restrict__ dstat, float* __restrict__ dO) {
  constexpr int EPL = D / kLanesPerKey;   // elements per lane (4 or 8)
  typedef RowPiece<EPL> RP;
  __shared__ float red[kThreads / 64][G];
  __shared__ float acc_s[kKeysPerRound][G * D + 4];
  const int s = blockIdx.x, nsplit = gridDim.x;
  const size_t bh = blockIdx.y;
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  const int head_rounds = (M + kKeysPerRound - 1) / kKeysPerRound;
  const int nrounds = (head_rounds - s + nsplit - 1) / nsplit;   // rounds s, s+ns, ...
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kg = tid / kLanesPerKey, slice = tid % kLanesPerKey;
  const bf16_t* kbase = kc + bh * (size_t)M * D + slice * EPL;
  const bf16_t* vbase = vc + bh * (size_t)M * D + slice * EPL;
  auto slot_of = [&](int rd) { return (s + rd * nsplit) * kKeysPerRound + kg; };

  // ring of PF rounds; slots past the cache re-read the last slot
  typename RP::raw_t kr[PF], vr[PF];
  auto issue = [&](int rd, int slot_) {
    const int kk = min(slot_of(rd), M - 1);
    kr[slot_] = RP::load(kbase + (size_t)kk * D);
    vr[slot_] = RP::load(vbase + (size_t)kk * D);
  };
#pragma unroll
  for (int u = 0; u < PF; ++u) issue(u, u);
  float qs[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float f[EPL];
    RP::unpack(RP::load(q + (size_t)(b * Hq + h * G + g) * D + slice * EPL), f);
#pragma unroll
    for (int e = 0; e < EPL; ++e) qs[g][e] = f[e] * c_log2;
  }
  float m[G], l[G], acc[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[g][e] = 0.f;
  }
  for (int rd0 = 0; rd0 < nrounds; rd0 += PF) {
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int rd = rd0 + u;
      if (rd < nrounds) {
        const int kk = slot_of(rd);
        const bool ok = kk < M;
        float kf[EPL], vf[EPL];
        RP::unpack(kr[u], kf);
        RP::unpack(vr[u], vf);
        issue(rd + PF, u);                       // refill the slot just consumed
        float lgs[G];
#pragma unroll
        for (int g = 0; g < G; ++g) {
          float a = 0.f;
#pragma unroll
          for (int e = 0; e < EPL; ++e) a = fmaf(qs[g][e], kf[e], a);
          lgs[g] = sum16(a);
        }
        if (ok && slice == 0) {                    // logits stored key-major: [bh][slot][g]
          float* dst = logits + ((bh * M) + kk) * (size_t)G;
#pragma unroll
          for (int g = 0; g < G; ++g) dst[g] = lgs[g];
        }
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const float lg = lgs[g];
          if (ok && lg > m[g] + 64.f) {            // first slot, or a much larger logit
            const float sc = __builtin_amdgcn_exp2f(m[g] - lg);
            l[g] *= sc;
#pragma unroll
            for (int e = 0; e < EPL; ++e) acc[g][e] *= sc;
            m[g] = lg;
          }
          const float p = ok ? __builtin_amdgcn_exp2f(lg - m[g]) : 0.f;
          l[g] += p;
#pragma unroll
          for (int e = 0; e < EPL; ++e) acc[g][e] = fmaf(p, vf[e], acc[g][e]);
        }
      }
    }
  }
  // block merge: common maximum per query head, rescale, sum through LDS
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float mx = m[g];
    for (int o = 16; o < 64; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    if (lane == 0) red[wave][g] = mx;
  }
  __syncthreads();
  float mb[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float mx = red[0][g];
#pragma unroll
    for (int w = 1; w < kThreads / 64; ++w) mx = fmaxf(mx, red[w][g]);
    mb[g] = mx;
  }
  __syncthreads();
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const float sc = m[g] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m[g] - mb[g]);
    float lv = slice == 0 ? l[g] * sc : 0.f;   // l is identical in the 16 lanes of a row
    for (int o = 16; o < 64; o <<= 1) lv += __shfl_xor(lv, o, 64);
    if (lane == 0) red[wave][g] = lv;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc_s[kg][g * D + slice * EPL + e] = acc[g][e] * sc;
  }
  __syncthreads();
  if (tid < G) {
    float lt = 0.f;
    for (int w = 0; w < kThreads / 64; ++w) lt += red[w][tid];
    dstat[(bh * nsplit + s) * G + tid] = make_float2(mb[tid], lt);
  }
  for (int c = tid; c < G * D; c += kThreads) {
    float a = 0.f;
#pragma unroll
    for (int k2 = 0; k2 < kKeysPerRound; ++k2) a += acc_s[k2][c];
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
  const float* lgb = logits + bh * (size_t)M * G;
  const int c0 = blockIdx.x * kCols, c1 = min(M, c0 + kCols);
  for (int j = c0 + tid; j < c1; j += kThreads) {
    float a = 0.f;
    for (int g = 0; g < G; ++g) a += __builtin_amdgcn_exp2f(lgb[(size_t)j * G + g] - lam[g]);
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
// at most one per round of slots.
template <int D, int G>
int split_count(int M, int BH) {
  static int resident = 0;
  if (!resident) {
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, decode_split<D, G, 8>, kThreads,
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
  const int rounds = (M + kKeysPerRound - 1) / kKeysPerRound;
  if (ns > rounds) ns = rounds;
  if (ns > kMaxSplit) ns = kMaxSplit;
  return ns < 1 ? 1 : ns;
}

template <int D, int G>
hipError_t launch_split(hipStream_t st, int BH, const void* q, const void* kc, const void* vc,
                        int Hq, int Hkv, int M, float c, float* logits, float2* dstat, float* dO,
                        int* ns) {
  *ns = split_count<D, G>(M, BH);
  return launch_kernel(K_DECODE_SPLIT, decode_split<D, G, 8>, dim3(*ns, BH), dim3(kThreads), st,
                       (const bf16_t*)q, (const bf16_t*)kc, (const bf16_t*)vc, Hq, Hkv, M, c,
                       logits, dstat, dO);
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
  int ns = 0;
  if (s.M > 0) {
    const int G = s.G();
    hipError_t e = hipErrorInvalidValue;
#define H2O_SPLIT(DD, GG) \
  e = launch_split<DD, GG>(st, s.BH(), q, kc, vc, s.Hq, s.Hkv, s.M, c, logits, dstat, dO, &ns)
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
