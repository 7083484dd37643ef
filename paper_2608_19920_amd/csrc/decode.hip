// Token generation (T = 1): the chunk is one query per query head, so the
// step streams the whole KV cache once and is bound by HBM bandwidth
// (Sec. "Sparse Attention. Key-Value Caching": N_q = 1, N_k = N_C).
//
//   split    block (split s, head bh) covers cache slots [s*kChunk, +kChunk).
//            Eight lanes share one key row: lane `slice` holds D/8 elements of
//            it, so each wave load reads eight consecutive rows (contiguous
//            bytes). All K and V loads of the block are issued before any
//            arithmetic. Logits (log2 domain) reduce over the 8 lanes with
//            DPP; the split's softmax partial (m, l, O-partial) per query head
//            is written out, and so are the logits for the column sums.
//   combine  block bh merges the splits with the chunk's own key (column M),
//            writes out and lse, and wsum[j] = sum_g exp2(logit_gj - lambda_g)
//            from the stored logits.
#include "internal.h"

namespace h2o {
namespace {

constexpr int kThreads = 256;
constexpr int kLanesPerKey = 8;
constexpr int kKeysPerRound = kThreads / kLanesPerKey;   // 32
constexpr int kRounds = 8;
constexpr int kChunk = kKeysPerRound * kRounds;          // 256 cache slots per block
constexpr int kMaxGD = 512;                              // G * D handled by these kernels

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, true));
}
// Sum over the 8 lanes of an aligned lane octet; every lane gets the total.
__device__ __forceinline__ float sum8(float v) {
  v += dpp<0xB1>(v);    // quad_perm [1,0,3,2]
  v += dpp<0x4E>(v);    // quad_perm [2,3,0,1]
  v += dpp<0x141>(v);   // row_half_mirror: lane l <-> 7-l within each octet
  return v;
}

__device__ __forceinline__ void unpack8(const uint4 w, float* f) {
  const uint32_t v[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    f[2 * e] = __uint_as_float(v[e] << 16);
    f[2 * e + 1] = __uint_as_float(v[e] & 0xFFFF0000u);
  }
}

template <int D, int G>
__global__ __launch_bounds__(kThreads) void decode_split(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    int Hq, int Hkv, int M, float c_log2, float* __restrict__ logits, float2* __restrict__ dstat,
    float* __restrict__ dO) {
  constexpr int EPL = D / kLanesPerKey;   // elements per lane (8 or 16)
  constexpr int VPL = EPL / 8;            // 16-byte vectors per lane
  __shared__ float red[kThreads / 64][G][2];
  __shared__ float acc_s[kKeysPerRound][G * D + 4];
  const int s = blockIdx.x, nsplit = gridDim.x;
  const size_t bh = blockIdx.y;
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  const int j0 = s * kChunk, n = min(kChunk, M - j0);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kg = tid / kLanesPerKey, slice = tid % kLanesPerKey;

  // Rows past the block's last slot re-read that slot (always in bounds) and
  // are masked below, so every load is unconditional and issued up front.
  uint4 kr[kRounds][VPL], vr[kRounds][VPL];
  const bf16_t* kbase = kc + (bh * M + j0) * (size_t)D + slice * EPL;
  const bf16_t* vbase = vc + (bh * M + j0) * (size_t)D + slice * EPL;
#pragma unroll
  for (int rd = 0; rd < kRounds; ++rd) {
    const int kk = min(rd * kKeysPerRound + kg, n - 1);
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      kr[rd][v] = *reinterpret_cast<const uint4*>(kbase + (size_t)kk * D + 8 * v);
      vr[rd][v] = *reinterpret_cast<const uint4*>(vbase + (size_t)kk * D + 8 * v);
    }
  }
  float qs[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const bf16_t* qp = q + (size_t)(b * Hq + h * G + g) * D + slice * EPL;
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      float f[8];
      unpack8(*reinterpret_cast<const uint4*>(qp + 8 * v), f);
#pragma unroll
      for (int e = 0; e < 8; ++e) qs[g][8 * v + e] = f[e] * c_log2;
    }
  }
  // logits of this lane octet's keys, every lane of the octet holds them
  float lg[kRounds][G];
#pragma unroll
  for (int rd = 0; rd < kRounds; ++rd) {
    float kf[EPL];
#pragma unroll
    for (int v = 0; v < VPL; ++v) unpack8(kr[rd][v], kf + 8 * v);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float a = 0.f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) a = fmaf(qs[g][e], kf[e], a);
      lg[rd][g] = sum8(a);
    }
  }
  // block max per query head
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float m = -INFINITY;
#pragma unroll
    for (int rd = 0; rd < kRounds; ++rd)
      if (rd * kKeysPerRound + kg < n) m = fmaxf(m, lg[rd][g]);
    for (int o = 8; o < 64; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    if (lane == 0) red[wave][g][0] = m;
  }
  __syncthreads();
  float mg[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float m = red[0][g][0];
#pragma unroll
    for (int w = 1; w < kThreads / 64; ++w) m = fmaxf(m, red[w][g][0]);
    mg[g] = m;
  }
  // probabilities, row sums, stored logits, O partial over this lane's keys
  float acc[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[g][e] = 0.f;
  float lsum[G];
#pragma unroll
  for (int g = 0; g < G; ++g) lsum[g] = 0.f;
#pragma unroll
  for (int rd = 0; rd < kRounds; ++rd) {
    const int kk = rd * kKeysPerRound + kg;
    const bool ok = kk < n;
    float vf[EPL];
#pragma unroll
    for (int v = 0; v < VPL; ++v) unpack8(vr[rd][v], vf + 8 * v);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float p = ok ? __builtin_amdgcn_exp2f(lg[rd][g] - mg[g]) : 0.f;
      lsum[g] += p;
      if (ok && slice == (g % kLanesPerKey))
        logits[(bh * G + g) * (size_t)M + j0 + kk] = lg[rd][g];
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[g][e] = fmaf(p, vf[e], acc[g][e]);
    }
  }
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float l = lsum[g];      // identical in the 8 lanes of an octet: reduce over octets
    for (int o = 8; o < 64; o <<= 1) l += __shfl_xor(l, o, 64);
    if (lane == 0) red[wave][g][1] = l;
  }
  // O partial: sum the per-octet accumulators through LDS
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc_s[kg][g * D + slice * EPL + e] = acc[g][e];
  __syncthreads();
  if (tid < G) {
    float l = 0.f;
    for (int w = 0; w < kThreads / 64; ++w) l += red[w][tid][1];
    dstat[(bh * nsplit + s) * G + tid] = make_float2(mg[tid], l);
  }
  for (int c = tid; c < G * D; c += kThreads) {
    float a = 0.f;
#pragma unroll 8
    for (int k2 = 0; k2 < kKeysPerRound; ++k2) a += acc_s[k2][c];
    dO[(bh * nsplit + s) * (size_t)(G * D) + c] = a;
  }
}

// Block (x, bh): merges the splits of head bh (every block recomputes the
// few per-head statistics), then writes wsum for columns [x*kCols, +kCols);
// block x == 0 also writes out and lse.
constexpr int kCols = 1024;

template <int D>
__global__ __launch_bounds__(kThreads) void decode_combine(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ kn, const bf16_t* __restrict__ vn,
    int Hq, int Hkv, int M, int nsplit, float c_log2, const float* __restrict__ logits,
    const float2* __restrict__ dstat, const float* __restrict__ dO, bf16_t* __restrict__ out,
    float* __restrict__ lse, float* __restrict__ wsum) {
  constexpr int kMaxG = kMaxGD / 64;
  __shared__ float lnew[kMaxG], lam[kMaxG], mfin[kMaxG], linv[kMaxG];
  const int G = Hq / Hkv;
  const size_t bh = blockIdx.y;
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
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
    for (int s = 0; s < nsplit; ++s) mx = fmaxf(mx, dstat[(bh * nsplit + s) * G + g].x);
    float L = __builtin_amdgcn_exp2f(lnew[g] - mx);
    for (int s = 0; s < nsplit; ++s) {
      const float2 st = dstat[(bh * nsplit + s) * G + g];
      L += st.y * __builtin_amdgcn_exp2f(st.x - mx);
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
      for (int s = 0; s < nsplit; ++s)
        a = fmaf(dO[(bh * nsplit + s) * (size_t)(G * D) + c],
                 __builtin_amdgcn_exp2f(dstat[(bh * nsplit + s) * G + g].x - mfin[g]), a);
      out[(size_t)(b * Hq + h * G + g) * D + dd] = f32_to_bf16(a * linv[g]);
    }
  }
  float* w = wsum + bh * (size_t)(M + 1);
  const int c0 = blockIdx.x * kCols, c1 = min(M, c0 + kCols);
  for (int j = c0 + tid; j < c1; j += kThreads) {
    float a = 0.f;
    for (int g = 0; g < G; ++g)
      a += __builtin_amdgcn_exp2f(logits[(bh * G + g) * (size_t)M + j] - lam[g]);
    w[j] = a;
  }
  if (blockIdx.x == 0 && tid == 0) {
    float a = 0.f;
    for (int g = 0; g < G; ++g) a += __builtin_amdgcn_exp2f(lnew[g] - lam[g]);
    w[M] = a;
  }
}

template <int D, int G>
void launch_split(dim3 grid, hipStream_t st, const void* q, const void* kc, const void* vc,
                  int Hq, int Hkv, int M, float c, float* logits, float2* dstat, float* dO) {
  decode_split<D, G><<<grid, kThreads, 0, st>>>((const bf16_t*)q, (const bf16_t*)kc,
                                                (const bf16_t*)vc, Hq, Hkv, M, c, logits, dstat,
                                                dO);
}

}  // namespace

int decode_nsplit(int M) { return (M + kChunk - 1) / kChunk; }
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
  const int ns = p.nsplit;
  if (s.M > 0) {
    dim3 grid(ns, s.BH());
    const int G = s.G();
    LaunchTimer lt(K_DECODE_SPLIT, st);
#define H2O_SPLIT(DD, GG) \
  launch_split<DD, GG>(grid, st, q, kc, vc, s.Hq, s.Hkv, s.M, c, logits, dstat, dO)
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
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  LaunchTimer lt(K_DECODE_COMBINE, st);
  const dim3 cgrid(s.M > 0 ? (s.M + kCols - 1) / kCols : 1, s.BH());
  if (s.d == 64)
    decode_combine<64><<<cgrid, kThreads, 0, st>>>(
        (const bf16_t*)q, (const bf16_t*)kn, (const bf16_t*)vn, s.Hq, s.Hkv, s.M, ns, c, logits,
        dstat, dO, (bf16_t*)out, lse, wsum);
  else
    decode_combine<128><<<cgrid, kThreads, 0, st>>>(
        (const bf16_t*)q, (const bf16_t*)kn, (const bf16_t*)vn, s.Hq, s.Hkv, s.M, ns, c, logits,
        dstat, dO, (bf16_t*)out, lse, wsum);
  return hipGetLastError();
}

}  // namespace h2o
