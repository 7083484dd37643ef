// Internal declarations shared by the libh2o translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stddef.h>
#include <stdint.h>

namespace h2o {

// ------------------------------------------------------------ element types
typedef uint16_t bf16_t;   // raw bfloat16 bits

__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}
// Round-to-nearest-even; inputs are finite here.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<bf16_t>(u >> 16);
}
__device__ __forceinline__ float load_elem(const float* p, size_t i) { return p[i]; }
__device__ __forceinline__ float load_elem(const bf16_t* p, size_t i) { return bf16_to_f32(p[i]); }
__device__ __forceinline__ void store_elem(float* p, size_t i, float v) { p[i] = v; }
__device__ __forceinline__ void store_elem(bf16_t* p, size_t i, float v) { p[i] = f32_to_bf16(v); }

// Buffer resource over [base, base + bytes): loads at offsets past the end
// return zero. Word 3 selects 32-bit data for gfx9-family buffers.
constexpr int kBufferFlags = 0x00020000;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           kBufferFlags);
}

// Order-preserving map of a float32 score to uint32 (a < b  <=>  key(a) <
// key(b)); both zeros map to the same key.
__device__ __forceinline__ uint32_t order_key(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u << 1) == 0u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// log2(e) and ln(2) in float32.
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// ----------------------------------------------------------- problem shape
// Two arrangements of the keys a chunk attends:
//  - chunk mode: [M cache slots, all visible || the T chunk keys, causal], the
//    chunk's keys and values passed separately (attend, then evict);
//  - cache mode (cache_only): the M cache slots alone, the chunk already
//    written into them, slot j visible to chunk query i iff
//    token_pos[j] - pos0 <= i (insert, then attend).
struct Shape {
  int B, Hq, Hkv, T, M, d;
  bool cache_only = false;
  int G() const { return Hq / Hkv; }
  int R() const { return G() * T; }      // packed query rows per KV head
  int Tk() const { return cache_only ? 0 : T; }   // chunk key columns
  int Nk() const { return M + Tk(); }    // key columns per KV head
  int BH() const { return B * Hkv; }
};

// Token positions of cache mode: tp = token_pos (nullptr in chunk mode), pos0
// = the position of the chunk's first query.
struct KeyPos {
  const int32_t* tp;
  int32_t pos0;
};

// The H2O score accumulation a column-sum pass can carry out for a chunk
// step (Eq. h2o-score): scores[bh][j] += wsum[bh][j] for the M cache slots,
// and, with copy non-null, the accumulated value also written to
// copy[bh][j] (the ranking input of the fused selection, which must not
// change while that kernel runs). scores null: no accumulation.
struct ScoreAcc {
  float* scores = nullptr;
  float* copy = nullptr;
};

// Packed row r of a KV head is (chunk position i = r / G, group member g = r % G).
// In chunk mode the keys a chunk position i may see are columns [0, M + i + 1).
// A partial-sum slot that covers packed rows [r0, r1) therefore sees key
// columns [0, kv_end) with kv_end = M + min(T-1, (r1-1)/G) + 1; with no chunk
// key columns (Tk = 0, cache mode) it is M.
__host__ __device__ __forceinline__ int kv_end_for_rows(int r1, int G, int T, int M, int Tk) {
  if (Tk == 0) return M;
  int i_max = (r1 - 1) / G;
  if (i_max > T - 1) i_max = T - 1;
  return M + i_max + 1;
}

// Cache-mode visibility of slot j to chunk position i (positions are compared
// in 64 bits, so any int32 token position works).
__device__ __forceinline__ bool pos_visible(int32_t tpj, int32_t pos0, int i) {
  return (long long)tpj - (long long)pos0 <= (long long)i;
}

__host__ __device__ __forceinline__ size_t align256_size(size_t n) { return (n + 255) & ~size_t(255); }

// ---------------------------------------------------------- workspace plan
// Layout of the scratch buffer used by h2o_sdpa_chunk. All offsets are byte
// offsets, 256-byte aligned.
struct Plan {
  int path;            // 0 = generic (float/bf16 VALU), 1 = bf16 MFMA, 2 = bf16 decode
  int rows_per_part;   // packed rows per colsum partial
  int nparts;          // partials per KV head
  int nsplit;          // key-range splits per row tile of the main pass (MFMA path)
  int nsplit_lse;      // key-range splits per row tile of the lse pass (MFMA path)
  int main_waves;      // waves per main-pass block, 4 or 8 (MFMA path)
  int lse_waves;       // waves per lse-pass block, 4 or 8 (MFMA path)
  int parts_ld;        // floats per colsum partial row (>= Nk)
  size_t off_stats;    // float2 (m, l) per (split, bh, row)  or lse per (bh,row)
  size_t off_parts;    // float colsum partials [nparts][BH][Nk]; decode: 1 KiB store sink
  size_t off_opart;    // float O partials [nsplit][BH][R][d] (nsplit > 1)
  size_t off_logits;   // decode: float logits [BH][G][Nk]
  size_t off_keys;     // float accumulated scores [BH][M], the ranking copy of a chunk step
  size_t bytes;
};
Plan make_plan(const Shape& s, int dtype);
int mfma_rows_per_wave();        // packed rows per wave of the MFMA kernels
int decode_max_split();      // largest split-block count per head of the decode kernels
bool decode_supports(int d, int G);   // (d, G) pairs the decode kernels handle

// ------------------------------------------------------------ kernel timing
// Identifiers of every kernel the library launches (for the timing hook).
enum KernelId {
  K_GENERIC_LSE = 0, K_GENERIC_MAIN, K_MFMA_LSE, K_MFMA_MAIN, K_SPLIT_REDUCE, K_COLSUM_REDUCE,
  K_ACCUMULATE, K_BOTTOMK, K_INSERT, K_DECODE_SPLIT, K_DECODE_COMBINE, K_ARGMIN_INSERT,
  K_DECODE_FINISH, K_KEYS, K_BWD_DQ, K_BWD_DKDV, K_KV_COPY, K_BWD_DOT, K_BWD_DQ_REDUCE,
  K_BOTTOMK_INSERT, K_COUNT
};
// While timing is switched on (h2o_debug_timing), kernels go out through
// hipExtLaunchKernel with a start and a stop event: the runtime stamps them
// with the kernel's own begin and end, so the pair measures the kernel and
// not the dispatch around it. timing_begin creates the pair (false when timing
// is off); timing_end queues it for h2o_debug_kernel_time.
bool timing_begin(hipEvent_t* a, hipEvent_t* b);
void timing_end(int kernel_id, hipEvent_t a, hipEvent_t b);

template <typename F, typename... Args>
hipError_t launch_kernel(int kernel_id, F kern, dim3 grid, dim3 block, hipStream_t st,
                         Args... args) {
  hipEvent_t a = nullptr, b = nullptr;
  if (timing_begin(&a, &b)) {
    hipExtLaunchKernelGGL(kern, grid, block, 0, st, a, b, 0, args...);
    const hipError_t e = hipGetLastError();
    timing_end(kernel_id, a, b);
    return e;
  }
  hipLaunchKernelGGL(kern, grid, block, 0, st, args...);
  return hipGetLastError();
}

// ------------------------------------------------------------- launchers
// Each returns hipSuccess or the launch error. They assume validated inputs.
// In cache mode (s.cache_only) kn and vn are unused and kp holds the token
// positions; in chunk mode kp.tp is nullptr.
// acc: the score accumulation of a chunk step, done in the column-sum pass
// (the bits of the separate accumulate kernel); none by default.
hipError_t launch_sdpa_generic(const Shape& s, const Plan& p, int dtype, const void* q,
                               const void* kc, const void* vc, const void* kn,
                               const void* vn, void* out, float* lse, float* wsum,
                               char* ws, float scale, KeyPos kp, hipStream_t st,
                               ScoreAcc acc = ScoreAcc{});
hipError_t launch_sdpa_mfma(const Shape& s, const Plan& p, const void* q, const void* kc,
                            const void* vc, const void* kn, const void* vn, void* out,
                            float* lse, float* wsum, char* ws, float scale, KeyPos kp,
                            hipStream_t st, ScoreAcc acc = ScoreAcc{});
// scores_acc (cache mode only, may be nullptr): scores to which the summed
// weights are added in the same pass (the accumulate of an insert-first step).
hipError_t launch_sdpa_decode(const Shape& s, const Plan& p, const void* q, const void* kc,
                              const void* vc, const void* kn, const void* vn, void* out,
                              float* lse, float* wsum, char* ws, float scale, KeyPos kp,
                              hipStream_t st, float* scores_acc = nullptr);
// T == 1, one call for the whole step: split kernel, then one block per head
// merges the splits, accumulates the scores, picks the slot and inserts.
hipError_t launch_decode_step(const Shape& s, const Plan& p, const void* q, void* kc, void* vc,
                              const void* kn, const void* vn, void* out, float* lse,
                              float* wsum, float* scores, int32_t* token_pos, int32_t* evict_idx,
                              int32_t pos0, char* ws, float scale, hipStream_t st);
// The same step as two calls: the attention (split, then out and lse) and
// the eviction (summed weights, accumulate, argmin, insert) from the split
// partials the attention left in the workspace. Same bits as the fused step.
hipError_t launch_decode_attend(const Shape& s, const Plan& p, const void* q, const void* kc,
                                const void* vc, const void* kn, const void* vn, void* out,
                                float* lse, char* ws, float scale, hipStream_t st);
hipError_t launch_decode_evict(const Shape& s, const Plan& p, const void* q, void* kc, void* vc,
                               const void* kn, const void* vn, float* wsum, float* scores,
                               int32_t* token_pos, int32_t* evict_idx, int32_t pos0, char* ws,
                               float scale, hipStream_t st);
// The insert-first step with the h2o ranking for T == 1 (cache mode), in two
// launches: the split kernel picks each head's evicted slot itself (the
// (score, slot)-smallest of the scores before the step), attends as if the
// chunk's key, value and position were already in that slot and writes them
// there; the combine adds the summed weights to the scores, the new slot's
// to 0. Same results as evict, insert, attend and accumulate in turn.
hipError_t launch_decode_step_insert_first(const Shape& s, const Plan& p, const void* q,
                                           void* kc, void* vc, float* scores, int32_t* token_pos,
                                           const void* kn, const void* vn, void* out, float* lse,
                                           float* wsum, int32_t* evict_idx, int32_t pos0,
                                           char* ws, float scale, hipStream_t st);
// acc: scores[bh][j] += wsum[bh][j] for j < M in the same pass (a chunk
// step's accumulation), with the optional copy.
hipError_t launch_colsum_reduce(const Shape& s, const Plan& p, const float* parts,
                                float* wsum, hipStream_t st, ScoreAcc acc = ScoreAcc{});
hipError_t launch_accumulate(float* scores, const float* wsum, int rows, int M, int T,
                             hipStream_t st);
hipError_t launch_bottomk(const float* scores, int rows, int M, int k, int32_t* idx,
                          hipStream_t st);
// Bottom-k of keys (row pitch M; not written while the kernel runs, and
// another array than scores) and the insert of the chunk (as launch_insert)
// in one launch, for the k that bottomk_insert_supported() accepts.
bool bottomk_insert_supported(int k);
hipError_t launch_bottomk_insert(const float* keys, float* scores, int32_t* token_pos, void* kc,
                                 void* vc, const void* kn, const void* vn, const float* wsum,
                                 int32_t* idx, int rows, int M, int T, int d, int k,
                                 int32_t pos0, int elem_bytes, hipStream_t st);
hipError_t launch_argmin_insert(void* kc, void* vc, float* scores, const float* keys,
                                int key_rows, int32_t* token_pos, const void* kn, const void* vn,
                                const float* wsum, int32_t* idx, int rows, int M, int T, int d,
                                int32_t pos0, int elem_bytes, hipStream_t st);
// Score variants: the ranked keys (h2o_norm per row, h2o_orig per kv head)
// and the broadcast of one index row per kv head over the batch.
hipError_t launch_norm_keys(const float* scores, const int32_t* token_pos, float* keys, int rows,
                            int M, int32_t t, hipStream_t st);
hipError_t launch_orig_keys(const float* scores, float* keys, int B, int Hkv, int M,
                            hipStream_t st);
hipError_t launch_broadcast_rows(const int32_t* src, int32_t* dst, int B, int n,
                                 hipStream_t st);
// The inserted slots take score wsum[row, M + i] (row pitch M + T), or 0
// when wsum is nullptr (insert before attending).
hipError_t launch_insert(void* kc, void* vc, float* scores, int32_t* token_pos,
                         const void* kn, const void* vn, const float* wsum,
                         const int32_t* idx, int rows, int M, int T, int d, int k,
                         int32_t pos0, int elem_bytes, hipStream_t st);

// Backward of the chunk attention (dq, dk, dv for the loss sum(dout * out));
// dot is the per-row scratch [BH][R]. Cache mode: kp.tp set, kn/vn/dkn/dvn
// unused.
hipError_t launch_sdpa_backward(const Shape& s, int dtype, const void* q, const void* kc,
                                const void* vc, const void* kn, const void* vn, KeyPos kp,
                                const float* lse, const void* dout, void* dq, void* dkc,
                                void* dvc, void* dkn, void* dvn, float* dot, float scale,
                                hipStream_t st);
// Workspace of the backward: D partials [ns_dot][BH][R] floats at offset 0
// (the VALU kernels use the first plane) and, with several, one more plane
// for their sum; then, when the dq pass is split, dq partials
// [ns_dq][BH][R][d] floats at off_part. dtype 0 (float32) has no splits.
struct BackwardPlan {
  int ns_dot, ns_dq;
  size_t off_part, bytes;
  int dq_waves;   // waves per block of the dq pass, 4 or 8
  int dot_waves;  // waves per block of the D pass, 4 or 8
};
int device_cus();   // compute units of the current device (256 where none answers)
BackwardPlan backward_plan(const Shape& s, int dtype);
// The same gradients on bf16 MFMA (bf16 data, d = 64 or 128): a rows pass
// for D_r, a rows pass for dq (plus the reduce of its split partials), a
// keys pass for dk and dv. ws: a workspace of backward_plan(s, 1).bytes.
hipError_t launch_sdpa_backward_mfma(const Shape& s, const void* q, const void* kc,
                                     const void* vc, const void* kn, const void* vn, KeyPos kp,
                                     const float* lse, const void* dout, void* dq, void* dkc,
                                     void* dvc, void* dkn, void* dvn, char* ws, float scale,
                                     hipStream_t st);
// rows[r, i] = cache[r, idx[r, i]] (gather) or cache[r, idx[r, i]] = rows[r, i]
// (scatter), `vecs` 16-byte vectors per cache row.
hipError_t launch_kv_copy(bool gather, void* cache, const int32_t* idx, void* rows, int nrows,
                          int M, int k, int vecs, hipStream_t st);

}  // namespace h2o
