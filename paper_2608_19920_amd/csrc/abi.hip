// C ABI of libh2o.so: argument validation, workspace plan, kernel dispatch.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/h2o.h"
#include "internal.h"

namespace h2o {
namespace {

thread_local std::string g_last_error;
std::atomic<int> g_forced_path{-1};

// Timing hook state: pending (kernel id, start, stop) event triples and the
// per-kernel totals folded in by h2o_debug_kernel_time.
std::atomic<bool> g_timing{false};
std::mutex g_timing_mu;
struct Pending { int id; hipEvent_t a, b; };
std::vector<Pending> g_pending;
double g_total_ms[K_COUNT];
long g_count[K_COUNT];

void fold_pending() {
  for (auto& p : g_pending) {
    float ms = 0.f;
    if (hipEventSynchronize(p.b) == hipSuccess && hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
      g_total_ms[p.id] += ms;
      g_count[p.id] += 1;
    }
    (void)hipEventDestroy(p.a);
    (void)hipEventDestroy(p.b);
  }
  g_pending.clear();
}

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int ok() {
  g_last_error.clear();
  return H2O_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Checks that a usable gfx950 device is current. Cached per device id.
int check_device() {
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || n <= 0) {
    (void)hipGetLastError();
    return fail(H2O_ENODEVICE, "no HIP device visible");
  }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(H2O_ENODEVICE, "hipGetDevice failed");
  static std::mutex mu;
  static int known[64] = {0};   // 0 unknown, 1 ok, 2 bad
  std::lock_guard<std::mutex> lk(mu);
  if (dev >= 0 && dev < 64 && known[dev] == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess)
      return fail(H2O_ENODEVICE, "hipGetDeviceProperties failed");
    known[dev] = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 2;
  }
  if (dev < 0 || dev >= 64 || known[dev] != 1)
    return fail(H2O_ENODEVICE, "device %d is not a gfx950 (MI355X) GPU", dev);
  return H2O_OK;
}

int check_shape(int B, int Hq, int Hkv, int T, int M, int d) {
  if (B < 1 || Hq < 1 || Hkv < 1) return fail(H2O_ESHAPE, "B, Hq, Hkv must be >= 1");
  if (Hq % Hkv) return fail(H2O_ESHAPE, "Hq (%d) must be a multiple of Hkv (%d)", Hq, Hkv);
  if (d != 64 && d != 128) return fail(H2O_ESHAPE, "head dim d=%d not supported (64 or 128)", d);
  if (T < 1) return fail(H2O_EINVAL, "chunk length T must be >= 1");
  if (M < 0) return fail(H2O_EINVAL, "cache length M must be >= 0");
  const long long nk = (long long)M + T;
  const long long rows = (long long)(Hq / Hkv) * T;
  if (nk * d >= (1ll << 30) || rows * d >= (1ll << 30) || (long long)B * Hq >= (1 << 24))
    return fail(H2O_ESHAPE, "shape too large for 32-bit per-head indexing");
  return H2O_OK;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Workspace of the score-variant eviction: the ranked keys, and for h2o_orig
// the per-head index rows before the broadcast over the batch.
size_t evict_workspace(int B, int Hkv, int M, int k, int policy) {
  if (policy == H2O_POLICY_NORM) return align256((size_t)B * Hkv * M * 4);
  if (policy == H2O_POLICY_ORIG)
    return align256((size_t)Hkv * M * 4) + align256((size_t)Hkv * k * 4);
  return 0;
}

}  // namespace

bool timing_begin(hipEvent_t* a, hipEvent_t* b) {
  if (!g_timing.load()) return false;
  if (hipEventCreate(a) != hipSuccess) return false;
  if (hipEventCreate(b) != hipSuccess) {
    (void)hipEventDestroy(*a);
    return false;
  }
  return true;
}

void timing_end(int kid, hipEvent_t a, hipEvent_t b) {
  std::lock_guard<std::mutex> lk(g_timing_mu);
  g_pending.push_back({kid, a, b});
}

// Compute units of the current device (cached per device; 256, the MI355X
// count, where no device answers, e.g. a size query on a host without one).
int device_cus() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    (void)hipGetLastError();
    return 256;
  }
  int n = cached[dev].load();
  if (n > 0) return n;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      n < 1) {
    (void)hipGetLastError();
    return 256;
  }
  cached[dev].store(n);
  return n;
}

Plan make_plan(const Shape& s, int dtype) {
  Plan p{};
  const size_t BH = s.BH(), R = s.R(), Nk = s.Nk();
  int path = dtype == H2O_BF16 ? 1 : 0;
  if (dtype == H2O_BF16 && s.T == 1 && decode_supports(s.d, s.G())) path = 2;
  const int forced = g_forced_path.load();
  if (dtype == H2O_BF16 && forced >= 0) path = forced;
  // the decode kernels need one query per head and an instantiated (d, G)
  if (path == 2 && (s.T != 1 || !decode_supports(s.d, s.G()))) path = 1;
  p.path = path;
  p.nsplit = 1;
  p.nsplit_lse = 1;
  p.parts_ld = (int)Nk;
  if (path == 1) {
    // Split the key range of each row tile when there are too few blocks to
    // fill the CUs (a round: the blocks resident at once; the main pass fits
    // two 4-wave or one 8-wave block per CU, the lighter lse pass four
    // 4-wave or two 8-wave blocks). Keep at least 8 key tiles per split.
    const long long ntiles = (Nk + 31) / 32;
    const long long cus = device_cus();
    auto pick = [&](long long nb, long long target, long long maxs) {
      long long ns = (target + nb - 1) / nb;
      if (ns > ntiles / 8) ns = ntiles / 8;
      if (ns > maxs) ns = maxs;
      return (int)(ns < 1 ? 1 : ns);
    };
    // main-pass blocks of `waves` waves: their row-tile count and split
    auto main_grid = [&](int waves, long long& nrt_w, int& ns_w) {
      const long long rows_w = (long long)waves * mfma_rows_per_wave();
      const long long round = cus * (8 / waves);
      nrt_w = ((long long)R + rows_w - 1) / rows_w;
      const long long nb = nrt_w * (long long)BH;
      ns_w = pick(nb, round, 8);
      // Between one and two rounds the second round is partly filled and
      // runs at the pace of its fullest CUs; halved blocks shorten it (896
      // row tiles of 128 rows at GQA 7:1: 1,150 -> 1,030 us for the pass,
      // 22 us for the O partials' reduce).
      if (ns_w == 1 && nb > round && nb < 2 * round && ntiles >= 16) ns_w = 2;
      return nb * ns_w % round == 0;   // whole rounds
    };
    // 8-wave blocks where they fill whole rounds (two blocks sharing a CU
    // advance unevenly; one block per CU leaves CUs idle in a partial round)
    long long nrt = 0;
    int ns = 1;
    p.main_waves = s.d == 128 && main_grid(8, nrt, ns) ? 8 : 4;
    if (p.main_waves == 4) main_grid(4, nrt, ns);
    p.nsplit = ns;
    // the lse pass: a round of 4-wave blocks (1,024 on 256 CUs), or of
    // 8-wave blocks where those fill whole rounds (long cache: the pass 580
    // against 610 us; more splits than one round's worth cost the main pass
    // as much in statistics reads)
    auto lse_grid = [&](int waves, int target, int& ns_w) {
      const long long rows_w = (long long)waves * mfma_rows_per_wave();
      const long long nb = (((long long)R + rows_w - 1) / rows_w) * (long long)BH;
      ns_w = pick(nb, target, 16);
      return nb * ns_w % (cus * (16 / waves)) == 0;
    };
    int nl = 1;
    p.lse_waves = s.d == 128 && lse_grid(8, (int)(2 * cus), nl) ? 8 : 4;
    if (p.lse_waves == 4) lse_grid(4, (int)(4 * cus), nl);
    p.nsplit_lse = nl;
    p.rows_per_part = p.main_waves * mfma_rows_per_wave();
    p.nparts = (int)nrt;
    p.parts_ld = (int)((Nk + 31) / 32 * 32);
  } else if (path == 2) {
    p.nsplit = s.M > 0 ? decode_max_split() : 0;   // capacity; the launch picks the count
    p.rows_per_part = 0;
    p.nparts = 0;
    size_t off = 0;
    p.off_stats = off;
    off = align256(off + (size_t)p.nsplit * BH * s.G() * sizeof(float) * 2);
    p.off_opart = off;
    off = align256(off + (size_t)p.nsplit * BH * s.G() * s.d * sizeof(float));
    p.off_logits = off;
    off = align256(off + BH * s.G() * (size_t)((s.M + 3) & ~3) * sizeof(float));
    p.off_parts = off;   // sink for the logit stores of masked slots (64 lanes x 16 B)
    off = align256(off + 64 * 16);
    p.bytes = off;
    return p;
  } else {
    p.rows_per_part = 64;
    p.nparts = (int)((R + 63) / 64);
  }
  size_t off = 0;
  p.off_stats = off;
  off = align256(off + (size_t)(p.nsplit_lse > p.nsplit ? p.nsplit_lse : p.nsplit) * BH * R *
                           sizeof(float) * 2);
  p.off_parts = off;
  off = align256(off + (size_t)p.nparts * BH * p.parts_ld * sizeof(float));
  p.off_opart = off;
  if (p.nsplit > 1) off = align256(off + (size_t)p.nsplit * BH * R * s.d * sizeof(float));
  p.off_logits = off;
  p.off_keys = off;
  off = align256(off + BH * (size_t)s.M * sizeof(float));
  p.bytes = off;
  return p;
}

namespace {

// Validation shared by the entry points that run the attention; fills *plan.
// In cache mode (token_pos non-null) the chunk's keys are in the cache:
// k_new and v_new are not read, and M >= 1.
int check_sdpa(const void* q, const void* k_cache, const void* v_cache, const void* k_new,
               const void* v_new, const void* out, const float* lse, const float* wsum,
               const void* workspace, size_t workspace_bytes, int B, int Hq, int Hkv, int T,
               int M, int d, float scale, int dtype, Plan* plan,
               const int32_t* token_pos = nullptr, size_t extra_bytes = 0) {
  const bool cache = token_pos != nullptr;
  if (dtype != H2O_F32 && dtype != H2O_BF16) return fail(H2O_EDTYPE, "dtype %d unknown", dtype);
  int rc = check_shape(B, Hq, Hkv, T, M, d);
  if (rc) return rc;
  if (cache && M < 1) return fail(H2O_EINVAL, "cache length M must be >= 1");
  if (!q || !out || !lse || !wsum || (!cache && (!k_new || !v_new)) ||
      (M > 0 && (!k_cache || !v_cache)))
    return fail(H2O_EINVAL, "null tensor pointer");
  if (!(std::isfinite(scale) && scale > 0.f)) return fail(H2O_EINVAL, "scale must be finite > 0");
  const void* ptrs[] = {q, out, lse, wsum, workspace, token_pos,
                        cache ? nullptr : k_new, cache ? nullptr : v_new};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return fail(H2O_EALIGN, "tensor pointer not 16-byte aligned");
  if (M > 0 && (!aligned16(k_cache) || !aligned16(v_cache)))
    return fail(H2O_EALIGN, "cache pointer not 16-byte aligned");
  const Shape s{B, Hq, Hkv, T, M, d, cache};
  *plan = make_plan(s, dtype);
  const size_t need = align256(plan->bytes) + extra_bytes;
  if (workspace_bytes < need || (need > 0 && !workspace))
    return fail(H2O_EWORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
  return H2O_OK;
}

// acc: the scores to which the summed weights of the M cache slots are added
// in the column-sum pass, with an optional copy (not on the decode path, whose
// T == 1 step has its own fused kernels).
hipError_t launch_sdpa(const Shape& s, const Plan& p, int dtype, const void* q,
                       const void* k_cache, const void* v_cache, const void* k_new,
                       const void* v_new, void* out, float* lse, float* wsum, void* workspace,
                       float scale, hipStream_t st, KeyPos kp = KeyPos{nullptr, 0},
                       ScoreAcc acc = ScoreAcc{}) {
  char* ws = reinterpret_cast<char*>(workspace);
  switch (p.path) {
    case 1:
      return launch_sdpa_mfma(s, p, q, k_cache, v_cache, k_new, v_new, out, lse, wsum, ws,
                              scale, kp, st, acc);
    case 2:
      return launch_sdpa_decode(s, p, q, k_cache, v_cache, k_new, v_new, out, lse, wsum, ws,
                                scale, kp, st);
    default:
      return launch_sdpa_generic(s, p, dtype, q, k_cache, v_cache, k_new, v_new, out, lse,
                                 wsum, ws, scale, kp, st, acc);
  }
}

// Validation of the eviction arguments shared by the entry points that evict.
int check_policy(int policy, const int32_t* token_pos) {
  if (policy != H2O_POLICY_H2O && policy != H2O_POLICY_NORM && policy != H2O_POLICY_ORIG)
    return fail(H2O_EINVAL, "policy %d unknown", policy);
  if (policy == H2O_POLICY_NORM && !token_pos)
    return fail(H2O_EINVAL, "h2o_norm needs token_pos (the slot ages)");
  return H2O_OK;
}

// Ranking of `policy` (norm ages against t), bottom-k and insert of the
// chunk; the inserted slots take score wsum[row, M+i] (row pitch M+T), or 0
// when wsum is nullptr. ews is the policy's workspace (evict_workspace()).
hipError_t launch_evict(int policy, void* k_cache, void* v_cache, float* scores,
                        int32_t* token_pos, const void* k_new, const void* v_new,
                        const float* wsum, int32_t* evict_idx, int B, int Hkv, int M, int T,
                        int d, int k, int32_t pos0, int32_t t, int eb, char* ews,
                        hipStream_t st) {
  const int rows = B * Hkv;
  const float* keys = scores;
  int key_rows = 0;
  float* wk = reinterpret_cast<float*>(ews);
  hipError_t e = hipSuccess;
  if (policy == H2O_POLICY_NORM) {
    e = launch_norm_keys(scores, token_pos, wk, rows, M, t, st);
    keys = wk;
  } else if (policy == H2O_POLICY_ORIG) {
    e = launch_orig_keys(scores, wk, B, Hkv, M, st);
    keys = wk;
    key_rows = Hkv;
  }
  if (e != hipSuccess) return e;
  if (k == 1)
    return launch_argmin_insert(k_cache, v_cache, scores, keys, key_rows, token_pos, k_new,
                                v_new, wsum, evict_idx, rows, M, T, d, pos0, eb, st);
  if (policy == H2O_POLICY_ORIG) {
    int32_t* head_idx = reinterpret_cast<int32_t*>(ews + align256((size_t)Hkv * M * 4));
    e = launch_bottomk(keys, Hkv, M, k, head_idx, st);
    if (e == hipSuccess) e = launch_broadcast_rows(head_idx, evict_idx, B, Hkv * k, st);
  } else {
    e = launch_bottomk(keys, rows, M, k, evict_idx, st);
  }
  if (e != hipSuccess) return e;
  return launch_insert(k_cache, v_cache, scores, token_pos, k_new, v_new, wsum, evict_idx, rows,
                       M, T, d, k, pos0, eb, st);
}

}  // namespace

}  // namespace h2o

using namespace h2o;

extern "C" {

const char* h2o_version(void) { return "h2o-mi355x 0.1 (gfx950)"; }

const char* h2o_last_error(void) { return g_last_error.c_str(); }

// Testing hook (not part of the stable ABI): force the SDPA kernel path for
// bf16 inputs. -1 = automatic, 0 = generic VALU, 1 = MFMA prefill, 2 = decode.
int h2o_debug_force_path(int path) {
  if (path < -1 || path > 2) return fail(H2O_EINVAL, "path must be -1..2");
  g_forced_path.store(path);
  return ok();
}

// Timing hook for benchmarks: while on, every kernel launch carries a start
// and a stop event stamped at the kernel's begin and end. Switching it (on or
// off) clears the totals.
int h2o_debug_timing(int on) {
  std::lock_guard<std::mutex> lk(g_timing_mu);
  fold_pending();
  for (int i = 0; i < K_COUNT; ++i) { g_total_ms[i] = 0.0; g_count[i] = 0; }
  g_timing.store(on != 0);
  return ok();
}

int h2o_debug_kernel_time(int kernel_id, double* total_ms, long* count) {
  if (kernel_id < 0 || kernel_id >= K_COUNT || !total_ms || !count)
    return fail(H2O_EINVAL, "kernel id out of range or null output");
  std::lock_guard<std::mutex> lk(g_timing_mu);
  fold_pending();
  *total_ms = g_total_ms[kernel_id];
  *count = g_count[kernel_id];
  return ok();
}

size_t h2o_workspace_bytes(int B, int Hq, int Hkv, int T, int M, int d, int dtype) {
  if (dtype != H2O_F32 && dtype != H2O_BF16) return 0;
  if (check_shape(B, Hq, Hkv, T, M, d) != H2O_OK) return 0;
  Shape s{B, Hq, Hkv, T, M, d};
  return make_plan(s, dtype).bytes;
}

int h2o_sdpa_chunk(const void* q, const void* k_cache, const void* v_cache, const void* k_new,
                   const void* v_new, void* out, float* lse, float* wsum, void* workspace,
                   size_t workspace_bytes, int B, int Hq, int Hkv, int T, int M, int d,
                   float scale, int dtype, void* stream) {
  Plan p;
  int rc = check_sdpa(q, k_cache, v_cache, k_new, v_new, out, lse, wsum, workspace,
                      workspace_bytes, B, Hq, Hkv, T, M, d, scale, dtype, &p);
  if (!rc) rc = check_device();
  if (rc) return rc;
  const Shape s{B, Hq, Hkv, T, M, d};
  hipError_t e = launch_sdpa(s, p, dtype, q, k_cache, v_cache, k_new, v_new, out, lse, wsum,
                             workspace, scale, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(H2O_ELAUNCH, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"

namespace h2o {
namespace {

enum StepPart { STEP_ALL, STEP_ATTEND, STEP_EVICT };

// h2o_chunk_step and its two halves: validation shared, then the kernels of
// the part asked for.
int chunk_step(StepPart part, const void* q, void* k_cache, void* v_cache, float* scores,
               int32_t* token_pos, const void* k_new, const void* v_new, void* out, float* lse,
               float* wsum, int32_t* evict_idx, void* workspace, size_t workspace_bytes, int B,
               int Hq, int Hkv, int T, int M, int d, float scale, int32_t pos0, int dtype,
               void* stream) {
  Plan p;
  int rc = check_sdpa(q, k_cache, v_cache, k_new, v_new, out, lse, wsum, workspace,
                      workspace_bytes, B, Hq, Hkv, T, M, d, scale, dtype, &p);
  if (rc) return rc;
  if (M < T) return fail(H2O_EINVAL, "cache length M (%d) must be >= T (%d)", M, T);
  if (!scores || !evict_idx) return fail(H2O_EINVAL, "null tensor pointer");
  if (!aligned16(scores) || !aligned16(evict_idx) || (token_pos && !aligned16(token_pos)))
    return fail(H2O_EALIGN, "tensor pointer not 16-byte aligned");
  rc = check_device();
  if (rc) return rc;
  const Shape s{B, Hq, Hkv, T, M, d};
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  char* ws = reinterpret_cast<char*>(workspace);
  hipError_t e = hipSuccess;
  if (p.path == 2) {
    if (part == STEP_ALL)
      e = launch_decode_step(s, p, q, k_cache, v_cache, k_new, v_new, out, lse, wsum, scores,
                             token_pos, evict_idx, pos0, ws, scale, st);
    else if (part == STEP_ATTEND)
      e = launch_decode_attend(s, p, q, k_cache, v_cache, k_new, v_new, out, lse, ws, scale, st);
    else
      e = launch_decode_evict(s, p, q, k_cache, v_cache, k_new, v_new, wsum, scores, token_pos,
                              evict_idx, pos0, ws, scale, st);
  } else {
    const int rows = B * Hkv, eb = dtype == H2O_F32 ? 4 : 2;
    // The whole step adds the summed weights to the scores in the column-sum
    // pass of the attention, which also leaves a copy of the accumulated
    // scores in the workspace for a selection and insert in one launch (the
    // copy is ranked, the scores are written). The evict half (after an
    // attend call) adds them on its own.
    const bool fused = part == STEP_ALL && T > 1 && bottomk_insert_supported(T);
    float* keys = reinterpret_cast<float*>(ws + p.off_keys);
    if (part != STEP_EVICT)
      e = launch_sdpa(s, p, dtype, q, k_cache, v_cache, k_new, v_new, out, lse, wsum, workspace,
                      scale, st, KeyPos{nullptr, 0},
                      ScoreAcc{part == STEP_ALL ? scores : nullptr, fused ? keys : nullptr});
    if (part != STEP_ATTEND) {
      if (e == hipSuccess && part == STEP_EVICT)
        e = launch_accumulate(scores, wsum, rows, M, T, st);
      if (e == hipSuccess && T == 1) {
        e = launch_argmin_insert(k_cache, v_cache, scores, scores, 0, token_pos, k_new, v_new,
                                 wsum, evict_idx, rows, M, T, d, pos0, eb, st);
      } else if (e == hipSuccess && fused) {
        e = launch_bottomk_insert(keys, scores, token_pos, k_cache, v_cache, k_new, v_new, wsum,
                                  evict_idx, rows, M, T, d, T, pos0, eb, st);
      } else if (e == hipSuccess) {
        e = launch_bottomk(scores, rows, M, T, evict_idx, st);
        if (e == hipSuccess)
          e = launch_insert(k_cache, v_cache, scores, token_pos, k_new, v_new, wsum, evict_idx,
                            rows, M, T, d, T, pos0, eb, st);
      }
    }
  }
  if (e != hipSuccess) return fail(H2O_ELAUNCH, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace
}  // namespace h2o

extern "C" {

int h2o_chunk_step(const void* q, void* k_cache, void* v_cache, float* scores,
                   int32_t* token_pos, const void* k_new, const void* v_new, void* out,
                   float* lse, float* wsum, int32_t* evict_idx, void* workspace,
                   size_t workspace_bytes, int B, int Hq, int Hkv, int T, int M, int d,
                   float scale, int32_t pos0, int dtype, void* stream) {
  return chunk_step(STEP_ALL, q, k_cache, v_cache, scores, token_pos, k_new, v_new, out, lse,
                    wsum, evict_idx, workspace, workspace_bytes, B, Hq, Hkv, T, M, d, scale,
                    pos0, dtype, stream);
}

}  // extern "C"

namespace h2o {
namespace {

// Scratch of h2o_chunk_step_noalloc, in place of a caller's workspace: one
// array on every device the library runs on, held until the process ends.
// In host code `scratch` names a host-side stand-in, not device memory:
// kernels get the address hipGetSymbolAddress returns for the current device.
constexpr size_t kScratchBytes = size_t(32) << 20;
static __device__ __align__(256) char scratch[kScratchBytes];

// Device address of `scratch` on the current device, looked up on the first
// call on that device (with it current) and kept.
int scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(H2O_ENODEVICE, "hipGetDevice failed");
  if (dev < 0 || dev >= 64) return fail(H2O_ENODEVICE, "device %d out of range", dev);
  static std::mutex mu;
  static void* addr[64] = {};
  std::lock_guard<std::mutex> lk(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      return fail(H2O_ELAUNCH, "hipGetSymbolAddress(scratch) failed: %s", hipGetErrorString(e));
    }
    addr[dev] = p;
  }
  *out = addr[dev];
  return H2O_OK;
}

}  // namespace
}  // namespace h2o

extern "C" {

size_t h2o_noalloc_scratch_bytes(void) { return kScratchBytes; }

int h2o_chunk_step_noalloc(const void* q, void* k_cache, void* v_cache, float* scores,
                           int32_t* token_pos, const void* k_new, const void* v_new, void* out,
                           float* lse, float* wsum, int32_t* evict_idx, int B, int Hq, int Hkv,
                           int T, int M, int d, float scale, int32_t pos0, int dtype,
                           void* stream) {
  if (dtype != H2O_F32 && dtype != H2O_BF16) return fail(H2O_EDTYPE, "dtype %d unknown", dtype);
  int rc = check_shape(B, Hq, Hkv, T, M, d);
  if (rc) return rc;
  const size_t need = make_plan(Shape{B, Hq, Hkv, T, M, d}, dtype).bytes;
  if (need > kScratchBytes)
    return fail(H2O_EWORKSPACE,
                "this shape needs %zu bytes of scratch; h2o_chunk_step_noalloc has %zu "
                "(use h2o_chunk_step with a workspace)", need, kScratchBytes);
  rc = check_device();
  if (rc) return rc;
  void* ws = nullptr;
  rc = scratch_address(&ws);
  if (rc) return rc;
  return chunk_step(STEP_ALL, q, k_cache, v_cache, scores, token_pos, k_new, v_new, out, lse,
                    wsum, evict_idx, ws, kScratchBytes, B, Hq, Hkv, T, M, d, scale, pos0, dtype,
                    stream);
}

int h2o_chunk_step_attend(const void* q, void* k_cache, void* v_cache, float* scores,
                          int32_t* token_pos, const void* k_new, const void* v_new, void* out,
                          float* lse, float* wsum, int32_t* evict_idx, void* workspace,
                          size_t workspace_bytes, int B, int Hq, int Hkv, int T, int M, int d,
                          float scale, int32_t pos0, int dtype, void* stream) {
  return chunk_step(STEP_ATTEND, q, k_cache, v_cache, scores, token_pos, k_new, v_new, out, lse,
                    wsum, evict_idx, workspace, workspace_bytes, B, Hq, Hkv, T, M, d, scale,
                    pos0, dtype, stream);
}

int h2o_chunk_step_evict(const void* q, void* k_cache, void* v_cache, float* scores,
                         int32_t* token_pos, const void* k_new, const void* v_new, void* out,
                         float* lse, float* wsum, int32_t* evict_idx, void* workspace,
                         size_t workspace_bytes, int B, int Hq, int Hkv, int T, int M, int d,
                         float scale, int32_t pos0, int dtype, void* stream) {
  return chunk_step(STEP_EVICT, q, k_cache, v_cache, scores, token_pos, k_new, v_new, out, lse,
                    wsum, evict_idx, workspace, workspace_bytes, B, Hq, Hkv, T, M, d, scale,
                    pos0, dtype, stream);
}

int h2o_accumulate_scores(float* scores, const float* wsum, int B, int Hkv, int M, int T,
                          void* stream) {
  if (B < 1 || Hkv < 1 || M < 0 || T < 0) return fail(H2O_ESHAPE, "bad sizes");
  if ((long long)B * Hkv * ((long long)M + T) >= (1ll << 40)) return fail(H2O_ESHAPE, "too large");
  if (M > 0 && (!scores || !wsum)) return fail(H2O_EINVAL, "null tensor pointer");
  if ((scores && !aligned16(scores)) || (wsum && !aligned16(wsum)))
    return fail(H2O_EALIGN, "tensor pointer not 16-byte aligned");
  int rc = check_device();
  if (rc) return rc;
  hipError_t e = launch_accumulate(scores, wsum, B * Hkv, M, T,
                                   reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(H2O_ELAUNCH, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

int h2o_bottomk(const float* scores, int rows, int M, int k, int32_t* idx_out, void* stream) {
  if (rows < 0 || M < 0 || k < 0 || k > M) return fail(H2O_EINVAL, "need rows >= 0, 0 <= k <= M");
  if ((long long)rows * M >= (1ll << 40)) return fail(H2O_ESHAPE, "too large");
  if (rows > 0 && k > 0 && (!scores || !idx_out)) return fail(H2O_EINVAL, "null tensor pointer");
  if ((scores && !aligned16(scores)) || (idx_out && !aligned16(idx_out)))
    return fail(H2O_EALIGN, "tensor pointer not 16-byte aligned");
  int rc = check_device();
  if (rc) return rc;
  hipError_t e = launch_bottomk(scores, rows, M, k, idx_out, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(H2O_ELAUNCH, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

size_t h2o_evict_workspace_bytes(int B, int Hkv, int M, int k, int policy) {
  if (B < 1 || Hkv < 1 || M < 0 || k < 0) return 0;
  return evict_workspace(B, Hkv, M, k, policy);
}

int h2o_evict_insert(void* k_cache, void* v_cache, float* scores, int32_t* token_pos,
                     const void* k_new, const void* v_new, const float* wsum, int32_t* evict_idx,
                     int B, int Hkv, int M, int T, int d, int k, int32_t pos0, int dtype,
                     void* stream) {
  return h2o_evict_insert_policy(k_cache, v_cache, scores, token_pos, k_new, v_new, wsum,
                                 evict_idx, B, Hkv, M, T, d, k, pos0, dtype, H2O_POLICY_H2O,
                                 nullptr, 0, stream);
}

int h2o_evict_insert_policy(void* k_cache, void* v_cache, float* scores, int32_t* token_pos,
                            const void* k_new, const void* v_new, const float* wsum,
                            int32_t* evict_idx, int B, int Hkv, int M, int T, int d, int k,
                            int32_t pos0, int dtype, int policy, void* workspace,
                            size_t workspace_bytes, void* stream) {
  if (dtype != H2O_F32 && dtype != H2O_BF16) return fail(H2O_EDTYPE, "dtype %d unknown", dtype);
  if (B < 1 || Hkv < 1) return fail(H2O_ESHAPE, "B, Hkv must be >= 1");
  if (d != 64 && d != 128) return fail(H2O_ESHAPE, "head dim d=%d not supported (64 or 128)", d);
  if (T < 1) return fail(H2O_EINVAL, "chunk length T must be >= 1");
  if (k != T) return fail(H2O_EINVAL, "k (%d) must equal T (%d): every chunk key is inserted", k, T);
  if (M < k) return fail(H2O_EINVAL, "cache length M (%d) must be >= k (%d)", M, k);
  if ((long long)B * Hkv * ((long long)M + T) * d >= (1ll << 40))
    return fail(H2O_ESHAPE, "too large");
  if (!k_cache || !v_cache || !scores || !k_new || !v_new || !wsum || !evict_idx)
    return fail(H2O_EINVAL, "null tensor pointer");
  int rc = check_policy(policy, token_pos);
  if (rc) return rc;
  const size_t need = evict_workspace(B, Hkv, M, k, policy);
  if (workspace_bytes < need)
    return fail(H2O_EWORKSPACE, "workspace %zu bytes, need %zu", workspace_bytes, need);
  if (need > 0 && !workspace) return fail(H2O_EINVAL, "null workspace");
  const void* ptrs[] = {k_cache, v_cache, scores, token_pos, k_new, v_new, wsum, evict_idx,
                        workspace};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return fail(H2O_EALIGN, "tensor pointer not 16-byte aligned");
  rc = check_device();
  if (rc) return rc;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int eb = dtype == H2O_F32 ? 4 : 2;
  // h2o_norm ranks after the chunk has been attended: t = pos0 + T
  hipError_t e = launch_evict(policy, k_cache, v_cache, scores, token_pos, k_new, v_new, wsum,
                              evict_idx, B, Hkv, M, T, d, k, pos0, pos0 + T, eb,
                              reinterpret_cast<char*>(workspace), st);
  if (e != hipSuccess) return fail(H2O_ELAUNCH, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

size_t h2o_cache_workspace_bytes(int B, int Hq, int Hkv, int T, int M, int d, int dtype,
                                 int policy) {
  if (dtype != H2O_F32 && dtype != H2O_BF16) return 0;
  if (check_shape(B, Hq, Hkv, T, M, d) != H2O_OK || M < 1) return 0;
  if (policy != H2O_POLICY_H2O && policy != H2O_POLICY_NORM && policy != H2O_POLICY_ORIG)
    return 0;
  const Shape s{B, Hq, Hkv, T, M, d, true};
  return align256(make_plan(s, dtype).bytes) + evict_workspace(B, Hkv, M, T, policy);
}

int h2o_sdpa_cache(const void* q, const void* k_cache, const void* v_cache,
                   const int32_t* token_pos, void* out, float* lse, float* wsum,
                   void* workspace, size_t workspace_bytes, int B, int Hq, int Hkv, int T, int M,
                   int d, float scale, int32_t pos0, int dtype, void* stream) {
  if (!token_pos) return fail(H2O_EINVAL, "null tensor pointer (token_pos)");
  Plan p;
  int rc = check_sdpa(q, k_cache, v_cache, nullptr, nullptr, out, lse, wsum, workspace,
                      workspace_bytes, B, Hq, Hkv, T, M, d, scale, dtype, &p, token_pos);
  if (!rc) rc = check_device();
  if (rc) return rc;
  const Shape s{B, Hq, Hkv, T, M, d, true};
  hipError_t e = launch_sdpa(s, p, dtype, q, k_cache, v_cache, nullptr, nullptr, out, lse, wsum,
                             workspace, scale, reinterpret_cast<hipStream_t>(stream),
                             KeyPos{token_pos, pos0});
  if (e != hipSuccess) return fail(H2O_ELAUNCH, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

int h2o_chunk_step_insert_first(const void* q, void* k_cache, void* v_cache, float* scores,
                                int32_t* token_pos, const void* k_new, const void* v_new,
                                void* out, float* lse, float* wsum, int32_t* evict_idx,
                                void* workspace, size_t workspace_bytes, int B, int Hq, int Hkv,
                                int T, int M, int d, float scale, int32_t pos0, int dtype,
                                int policy, void* stream) {
  if (!token_pos || !scores || !evict_idx || !k_new || !v_new)
    return fail(H2O_EINVAL, "null tensor pointer");
  if (M < T) return fail(H2O_EINVAL, "cache length M (%d) must be >= T (%d)", M, T);
  int rc = check_policy(policy, token_pos);
  if (rc) return rc;
  const size_t ews_bytes = evict_workspace(B, Hkv, M, T, policy);
  Plan p;
  rc = check_sdpa(q, k_cache, v_cache, nullptr, nullptr, out, lse, wsum, workspace,
                  workspace_bytes, B, Hq, Hkv, T, M, d, scale, dtype, &p, token_pos, ews_bytes);
  if (rc) return rc;
  if (!aligned16(scores) || !aligned16(evict_idx) || !aligned16(k_new) || !aligned16(v_new))
    return fail(H2O_EALIGN, "tensor pointer not 16-byte aligned");
  rc = check_device();
  if (rc) return rc;
  const Shape s{B, Hq, Hkv, T, M, d, true};
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  char* ws = reinterpret_cast<char*>(workspace);
  const int eb = dtype == H2O_F32 ? 4 : 2;
  // T == 1 on the decode kernels with the h2o ranking: the split kernel picks
  // and fills the slot itself (two launches, same results)
  if (p.path == 2 && policy == H2O_POLICY_H2O) {
    const hipError_t e = launch_decode_step_insert_first(s, p, q, k_cache, v_cache, scores,
                                                         token_pos, k_new, v_new, out, lse,
                                                         wsum, evict_idx, pos0, ws, scale, st);
    if (e != hipSuccess)
      return fail(H2O_ELAUNCH, "kernel launch failed: %s", hipGetErrorString(e));
    return ok();
  }
  // rank by the scores after pos0 tokens, then write the chunk into the
  // chosen slots with score 0 and positions pos0 + i
  hipError_t e = launch_evict(policy, k_cache, v_cache, scores, token_pos, k_new, v_new, nullptr,
                              evict_idx, B, Hkv, M, T, d, T, pos0, pos0, eb,
                              ws + align256(p.bytes), st);
  if (e == hipSuccess && p.path == 2) {
    // the decode combine adds the summed weights to the scores itself
    e = launch_sdpa_decode(s, p, q, k_cache, v_cache, nullptr, nullptr, out, lse, wsum, ws,
                           scale, KeyPos{token_pos, pos0}, st, scores);
  } else if (e == hipSuccess) {
    // the attention over the cache adds the summed weights to the scores in
    // its column-sum pass
    e = launch_sdpa(s, p, dtype, q, k_cache, v_cache, nullptr, nullptr, out, lse, wsum, ws,
                    scale, st, KeyPos{token_pos, pos0}, ScoreAcc{scores, nullptr});
  }
  if (e != hipSuccess) return fail(H2O_ELAUNCH, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

size_t h2o_backward_workspace_bytes(int B, int Hq, int Hkv, int T, int M, int d, int dtype) {
  if (dtype != H2O_F32 && dtype != H2O_BF16) return 0;
  if (check_shape(B, Hq, Hkv, T, M, d) != H2O_OK) return 0;
  const Shape s{B, Hq, Hkv, T, M, d};
  return backward_plan(s, dtype == H2O_BF16 ? 1 : 0).bytes;
}

int h2o_sdpa_chunk_backward(const void* q, const void* k_cache, const void* v_cache,
                            const void* k_new, const void* v_new, const int32_t* token_pos,
                            const float* lse, const void* dout, void* dq,
                            void* dk_cache, void* dv_cache, void* dk_new, void* dv_new,
                            void* workspace, size_t workspace_bytes, int B, int Hq, int Hkv,
                            int T, int M, int d, float scale, int32_t pos0, int dtype,
                            void* stream) {
  if (dtype != H2O_F32 && dtype != H2O_BF16) return fail(H2O_EDTYPE, "dtype %d unknown", dtype);
  int rc = check_shape(B, Hq, Hkv, T, M, d);
  if (rc) return rc;
  const bool cache = token_pos != nullptr;
  if (cache && M < 1) return fail(H2O_EINVAL, "cache length M must be >= 1");
  if (!(std::isfinite(scale) && scale > 0.f)) return fail(H2O_EINVAL, "scale must be finite > 0");
  if (!q || !lse || !dout || !dq ||
      (M > 0 && (!k_cache || !v_cache || !dk_cache || !dv_cache)) ||
      (!cache && (!k_new || !v_new || !dk_new || !dv_new)))
    return fail(H2O_EINVAL, "null tensor pointer");
  const void* ptrs[] = {q, k_cache, v_cache, lse, dout, dq, dk_cache, dv_cache, workspace,
                        token_pos, cache ? nullptr : k_new, cache ? nullptr : v_new,
                        cache ? nullptr : dk_new, cache ? nullptr : dv_new};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return fail(H2O_EALIGN, "tensor pointer not 16-byte aligned");
  const size_t need = h2o_backward_workspace_bytes(B, Hq, Hkv, T, M, d, dtype);
  if (workspace_bytes < need || !workspace)
    return fail(H2O_EWORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
  rc = check_device();
  if (rc) return rc;
  const Shape s{B, Hq, Hkv, T, M, d, cache};
  // bf16 runs on the MFMA kernels unless the generic path is forced
  const bool mfma = dtype == H2O_BF16 && g_forced_path.load() != 0;
  const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const KeyPos kp{token_pos, pos0};
  hipError_t e =
      mfma ? launch_sdpa_backward_mfma(s, q, k_cache, v_cache, k_new, v_new, kp, lse, dout, dq,
                                       dk_cache, dv_cache, dk_new, dv_new,
                                       reinterpret_cast<char*>(workspace), scale, st)
           : launch_sdpa_backward(s, dtype, q, k_cache, v_cache, k_new, v_new, kp, lse, dout,
                                  dq, dk_cache, dv_cache, dk_new, dv_new,
                                  reinterpret_cast<float*>(workspace), scale, st);
  if (e != hipSuccess) return fail(H2O_ELAUNCH, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

namespace {
int kv_copy_call(bool gather, void* cache, const int32_t* idx, void* rows, int B, int Hkv, int M,
                 int k, int d, int dtype, void* stream) {
  if (dtype != H2O_F32 && dtype != H2O_BF16) return fail(H2O_EDTYPE, "dtype %d unknown", dtype);
  if (B < 1 || Hkv < 1 || M < 1 || k < 0 || k > M)
    return fail(H2O_ESHAPE, "need B, Hkv, M >= 1 and 0 <= k <= M");
  if (d != 64 && d != 128) return fail(H2O_ESHAPE, "head dim d=%d not supported (64 or 128)", d);
  if ((long long)B * Hkv * M * d >= (1ll << 40)) return fail(H2O_ESHAPE, "too large");
  if (k > 0 && (!cache || !idx || !rows)) return fail(H2O_EINVAL, "null tensor pointer");
  if ((cache && !aligned16(cache)) || (idx && !aligned16(idx)) || (rows && !aligned16(rows)))
    return fail(H2O_EALIGN, "tensor pointer not 16-byte aligned");
  int rc = check_device();
  if (rc) return rc;
  const int eb = dtype == H2O_F32 ? 4 : 2;
  hipError_t e = launch_kv_copy(gather, cache, idx, rows, B * Hkv, M, k, d * eb / 16,
                                reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(H2O_ELAUNCH, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}
}  // namespace

int h2o_kv_gather(const void* cache, const int32_t* idx, void* delta, int B, int Hkv, int M,
                  int k, int d, int dtype, void* stream) {
  return kv_copy_call(true, const_cast<void*>(cache), idx, delta, B, Hkv, M, k, d, dtype,
                      stream);
}

int h2o_kv_scatter(void* cache, const int32_t* idx, const void* src, int B, int Hkv, int M, int k,
                   int d, int dtype, void* stream) {
  return kv_copy_call(false, cache, idx, const_cast<void*>(src), B, Hkv, M, k, d, dtype, stream);
}

}  // extern "C"
