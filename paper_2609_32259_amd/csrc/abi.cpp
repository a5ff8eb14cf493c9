// C ABI of the transfer path: argument validation, dispatch to the kernel
// launchers, error reporting and the kernel-timing profiler.  Nothing here
// touches the HIP runtime before all host-side checks of a call have passed,
// and loading the library initializes nothing.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "heterofold.h"
#include "hf_internal.h"

namespace {

thread_local std::string g_err;

int32_t fail(int32_t status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return status;
}

int32_t ok() {
  g_err.clear();
  return HF_OK;
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// ---------------------------------------------------------------------------
// Profiler: HIP event pairs around kernel launches, per kernel id.
// ---------------------------------------------------------------------------
struct EventPair {
  int kernel;
  hipEvent_t start, stop;
};

struct Profiler {
  std::mutex mu;
  bool on = false;
  std::vector<EventPair> pending;
  double total_ms[HF_KERNEL_COUNT] = {};
  int64_t launches[HF_KERNEL_COUNT] = {};
  std::vector<float> samples[HF_KERNEL_COUNT];  // per-launch ms, at most kMaxSamples each
};

constexpr size_t kMaxSamples = 4096;

Profiler& prof() {
  static Profiler p;
  return p;
}

// Scope that records a start event before and a stop event after the launches
// made while it lives, when the profiler is on.
class TimedLaunch {
 public:
  TimedLaunch(int kernel, hipStream_t s, bool enabled = true) : kernel_(kernel), s_(s) {
    if (!enabled) return;
    Profiler& p = prof();
    std::lock_guard<std::mutex> g(p.mu);
    if (!p.on) return;
    if (hipEventCreate(&ev_.start) != hipSuccess) return;
    if (hipEventCreate(&ev_.stop) != hipSuccess) {
      (void)hipEventDestroy(ev_.start);
      return;
    }
    if (hipEventRecord(ev_.start, s_) != hipSuccess) {
      (void)hipEventDestroy(ev_.start);
      (void)hipEventDestroy(ev_.stop);
      return;
    }
    active_ = true;
  }
  ~TimedLaunch() {
    if (!active_) return;
    Profiler& p = prof();
    std::lock_guard<std::mutex> g(p.mu);
    if (hipEventRecord(ev_.stop, s_) != hipSuccess) {
      (void)hipEventDestroy(ev_.start);
      (void)hipEventDestroy(ev_.stop);
      return;
    }
    ev_.kernel = kernel_;
    p.pending.push_back(ev_);
  }

 private:
  int kernel_;
  hipStream_t s_;
  EventPair ev_{};
  bool active_ = false;
};

// Collect finished event pairs into the totals (waits for them).
int32_t drain_profiler(Profiler& p) {
  for (EventPair& e : p.pending) {
    float ms = 0.f;
    hipError_t st = hipEventSynchronize(e.stop);
    if (st == hipSuccess) st = hipEventElapsedTime(&ms, e.start, e.stop);
    (void)hipEventDestroy(e.start);
    (void)hipEventDestroy(e.stop);
    if (st != hipSuccess) {
      p.pending.clear();
      return fail(HF_ERR_HIP, "profiler event: %s", hipGetErrorString(st));
    }
    p.total_ms[e.kernel] += ms;
    p.launches[e.kernel] += 1;
    if (p.samples[e.kernel].size() < kMaxSamples) p.samples[e.kernel].push_back(ms);
  }
  p.pending.clear();
  return HF_OK;
}

int32_t hip_fail(hipError_t e, const char* what) {
  return fail(HF_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Per-sequence counts from [B+1] prefix sums.
int32_t check_prefix(const char* name, int32_t B, const int32_t* cu) {
  if (cu[0] != 0) return fail(HF_ERR_SHAPE, "%s[0] must be 0", name);
  for (int b = 0; b < B; ++b)
    if (cu[b + 1] < cu[b]) return fail(HF_ERR_SHAPE, "%s is not non-decreasing at %d", name, b);
  return HF_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int32_t check_desc(const char* name, const hf_kv_desc* d) {
  if (!d) return fail(HF_ERR_NULL, "%s descriptor is NULL", name);
  if (!d->ptr) return fail(HF_ERR_NULL, "%s->ptr is NULL", name);
  if (d->dtype != HF_F32 && d->dtype != HF_BF16) return fail(HF_ERR_DTYPE, "%s->dtype %d unknown", name, d->dtype);
  if (d->L < 1 || d->H < 1 || d->d_h < 2 || (d->d_h & 1) || d->T_cap < 0)
    return fail(HF_ERR_SHAPE, "%s: need L>=1, H>=1, even d_h>=2, T_cap>=0", name);
  const int64_t vec = d->dtype == HF_BF16 ? 8 : 4;  // elements per 16 bytes
  if (!aligned16(d->ptr)) return fail(HF_ERR_SHAPE, "%s->ptr is not 16-byte aligned", name);
  const int64_t st[5] = {d->stride_b, d->stride_l, d->stride_c, d->stride_h, d->stride_t};
  for (int i = 0; i < 5; ++i)
    if (st[i] < 0 || st[i] % vec) return fail(HF_ERR_SHAPE, "%s: strides must be >= 0 and keep rows 16-byte aligned", name);
  if (d->d_h % vec) return fail(HF_ERR_SHAPE, "%s: d_h must be a multiple of %lld", name, (long long)vec);
  if (d->stride_t < d->d_h) return fail(HF_ERR_SHAPE, "%s: stride_t < d_h", name);
  return HF_OK;
}

}  // namespace

extern "C" {

const char* hf_last_error(void) { return g_err.c_str(); }

int32_t hf_version(void) { return HF_VERSION; }

int32_t hf_validate_offsets_host(int32_t T, const int32_t* beg, const int32_t* end) {
  if (T < 0) return fail(HF_ERR_SHAPE, "T must be >= 0");
  if (T > 0 && (!beg || !end)) return fail(HF_ERR_NULL, "beg/end is NULL");
  for (int32_t t = 0; t < T; ++t) {
    if (beg[t] < 0 || beg[t] > end[t])
      return fail(HF_ERR_OFFSETS, "token %d: need 0 <= beg <= end (got %d, %d)", t, beg[t], end[t]);
    if (t + 1 < T && end[t] > beg[t + 1])
      return fail(HF_ERR_OFFSETS, "tokens %d and %d overlap or are out of order", t, t + 1);
  }
  return ok();
}

int64_t hf_alignment_nnz_capacity(int32_t B, const int32_t* s_len, const int32_t* r_len,
                                  int32_t mode) {
  if (B < 1 || B > HF_MAX_BATCH || !s_len || !r_len) {
    fail(HF_ERR_SHAPE, "need 1 <= B <= %d and non-NULL lengths", HF_MAX_BATCH);
    return -1;
  }
  if (mode != HF_ALIGN_OVERLAP && mode != HF_ALIGN_TA) {
    fail(HF_ERR_MODE, "alignment mode %d unknown", mode);
    return -1;
  }
  int64_t cap = 0;
  for (int b = 0; b < B; ++b) {
    if (s_len[b] < 0 || r_len[b] < 0) {
      fail(HF_ERR_SHAPE, "negative length in sequence %d", b);
      return -1;
    }
    cap += mode == HF_ALIGN_TA ? (int64_t)r_len[b] : (int64_t)s_len[b] + 2 * (int64_t)r_len[b];
  }
  ok();
  return cap;
}

size_t hf_alignment_workspace_bytes(int32_t B, const int32_t* r_cu) {
  if (B < 1 || B > HF_MAX_BATCH || !r_cu) return 0;
  int nblk = 0;
  for (int b = 0; b < B; ++b) nblk += (r_cu[b + 1] - r_cu[b] + hf::kAlignBlock - 1) / hf::kAlignBlock;
  return hf::align_workspace_bytes(nblk);
}

int32_t hf_build_alignment(int32_t B, const int32_t* s_cu, const int32_t* r_cu,
                           const int32_t* s_beg, const int32_t* s_end, const int32_t* r_beg,
                           const int32_t* r_end, int32_t mode, int32_t* row_ptr, int32_t* col,
                           int32_t* num, int32_t* den, int64_t nnz_capacity, void* workspace,
                           size_t workspace_bytes, void* stream) {
  if (B < 1 || B > HF_MAX_BATCH) return fail(HF_ERR_SHAPE, "B=%d outside [1, %d]", B, HF_MAX_BATCH);
  if (!s_cu || !r_cu) return fail(HF_ERR_NULL, "s_cu / r_cu is NULL");
  if (mode != HF_ALIGN_OVERLAP && mode != HF_ALIGN_TA) return fail(HF_ERR_MODE, "alignment mode %d unknown", mode);
  int32_t st;
  if ((st = check_prefix("s_cu", B, s_cu)) || (st = check_prefix("r_cu", B, r_cu))) return st;
  const int64_t nS = s_cu[B], nR = r_cu[B];
  for (int b = 0; b < B; ++b)
    if (r_cu[b + 1] > r_cu[b] && s_cu[b + 1] == s_cu[b])
      return fail(HF_ERR_SHAPE, "sequence %d has receiver tokens but no sender tokens", b);
  if (!row_ptr) return fail(HF_ERR_NULL, "row_ptr is NULL");
  if (nR > 0 && (!r_beg || !r_end || !den)) return fail(HF_ERR_NULL, "receiver spans / den is NULL");
  if (nS > 0 && (!s_beg || !s_end)) return fail(HF_ERR_NULL, "sender spans are NULL");
  if (nR > 0 && (!col || !num)) return fail(HF_ERR_NULL, "col / num is NULL");
  if (nS + 2 * nR > INT32_MAX) return fail(HF_ERR_SHAPE, "batch too large for int32 CSR offsets");
  const int64_t need = mode == HF_ALIGN_TA ? nR : nS + 2 * nR;  // hf_alignment_nnz_capacity
  if (nnz_capacity < need)
    return fail(HF_ERR_CAPACITY, "nnz_capacity %lld < required %lld", (long long)nnz_capacity, (long long)need);

  hf::AlignArgs a;
  std::memset(&a, 0, sizeof a);
  int nblk = 0;
  for (int b = 0; b < B; ++b) {
    a.blk_start[b] = nblk;
    a.s0[b] = s_cu[b];
    a.Ts[b] = s_cu[b + 1] - s_cu[b];
    a.r0[b] = r_cu[b];
    a.Tr[b] = r_cu[b + 1] - r_cu[b];
    nblk += (a.Tr[b] + hf::kAlignBlock - 1) / hf::kAlignBlock;
  }
  a.blk_start[B] = nblk;
  const size_t ws_need = hf::align_workspace_bytes(nblk);
  if (!workspace) return fail(HF_ERR_NULL, "workspace is NULL");
  if (workspace_bytes < ws_need)
    return fail(HF_ERR_CAPACITY, "workspace %zu bytes < required %zu", workspace_bytes, ws_need);
  if (!aligned16(workspace)) return fail(HF_ERR_SHAPE, "workspace is not 16-byte aligned");
  const size_t n = (size_t)(nblk > 0 ? nblk : 1);
  char* w = static_cast<char*>(workspace);
  a.blk_sum = reinterpret_cast<long long*>(w);
  w += align_up(n * sizeof(long long), 256);
  a.blk_off = reinterpret_cast<long long*>(w);
  w += align_up(n * sizeof(long long), 256);
  a.blk_last = reinterpret_cast<int32_t*>(w);
  w += align_up(n * sizeof(int32_t), 256);
  a.blk_carry = reinterpret_cast<int32_t*>(w);
  a.s_beg = s_beg;
  a.s_end = s_end;
  a.r_beg = r_beg;
  a.r_end = r_end;
  a.row_ptr = row_ptr;
  a.col = col;
  a.num = num;
  a.den = den;
  a.cap = nnz_capacity;
  a.mode = mode;
  a.B = B;
  a.nblk = nblk;
  a.total_rows = (int32_t)nR;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  {
    TimedLaunch t(HF_KERNEL_ALIGNMENT, s);
    e = hf::launch_alignment(a, s);
  }
  if (e != hipSuccess) return hip_fail(e, "alignment launch");
  return ok();
}

int32_t hf_build_layer_map(int32_t L_s, int32_t L_r, int32_t mode, int32_t* lo, int32_t* hi,
                           int32_t* rem, int32_t* den) {
  if (mode != HF_LAYERS_INTERP2) return fail(HF_ERR_MODE, "layer mode %d unknown", mode);
  if (L_s < 1 || L_r < 1) return fail(HF_ERR_SHAPE, "layer counts must be >= 1");
  if (!lo || !hi || !rem || !den) return fail(HF_ERR_NULL, "output table is NULL");
  for (int32_t j = 0; j < L_r; ++j) {
    if (L_r == 1) {
      lo[j] = hi[j] = rem[j] = 0;
      den[j] = 1;
      continue;
    }
    const int64_t n = (int64_t)j * (L_s - 1), d = L_r - 1;
    lo[j] = (int32_t)(n / d);
    rem[j] = (int32_t)(n % d);
    den[j] = (int32_t)d;
    hi[j] = std::min(lo[j] + 1, L_s - 1);
  }
  return ok();
}

int32_t hf_build_layer_taps(int32_t L_s, int32_t L_r, int32_t* taps) {
  if (L_s < 1 || L_r < 1) return fail(HF_ERR_SHAPE, "layer counts must be >= 1");
  if (!taps) return fail(HF_ERR_NULL, "output table is NULL");
  for (int32_t j = 0; j < L_r; ++j) {
    // pi = round(j (L_s-1) / (L_r-1)), ties to even, on exact integers
    int64_t pi = 0;
    if (L_r > 1) {
      const int64_t n = (int64_t)j * (L_s - 1), d = L_r - 1;
      pi = n / d;
      const int64_t r2 = 2 * (n % d);
      if (r2 > d || (r2 == d && (pi & 1))) ++pi;
    }
    for (int t = 0; t < 3; ++t) {
      const int64_t v = pi + 4 * (t - 1);
      taps[3 * j + t] = (int32_t)std::min<int64_t>(std::max<int64_t>(v, 0), L_s - 1);
    }
  }
  return ok();
}

size_t hf_packed_maps_bytes(int32_t L_r, int32_t d_r, int32_t d_in, int32_t dtype) {
  if (L_r < 1 || d_r < 1 || d_in < 1) return 0;
  const size_t el = dtype == HF_BF16 ? 2 : (dtype == HF_F32 ? 4 : 0);
  if (el == 0) return 0;
  return HF_PACKED_HEADER_BYTES + (size_t)L_r * 2 * (size_t)d_r * (size_t)d_in * el;
}

int32_t hf_pack_maps(int32_t L_r, int32_t d_r, int32_t d_in, int32_t dtype, const void* A,
                     void* A_packed, void* stream) {
  if (dtype != HF_F32 && dtype != HF_BF16) return fail(HF_ERR_DTYPE, "dtype %d unknown", dtype);
  if (L_r < 1 || L_r > HF_MAX_LAYERS || d_r < 1 || d_in < 1)
    return fail(HF_ERR_SHAPE, "need 1 <= L_r <= %d, d_r >= 1, d_in >= 1", HF_MAX_LAYERS);
  if (dtype == HF_BF16 && (d_in % 16 || d_r % 32))
    return fail(HF_ERR_SHAPE, "bf16 maps need d_in %% 16 == 0 and d_r %% 32 == 0");
  if (dtype == HF_F32 && (d_in % 4))
    return fail(HF_ERR_SHAPE, "fp32 maps need d_in %% 4 == 0");
  if (!A || !A_packed) return fail(HF_ERR_NULL, "A / A_packed is NULL");
  if (!aligned16(A) || !aligned16(A_packed)) return fail(HF_ERR_SHAPE, "A / A_packed not 16-byte aligned");
  const size_t bytes = hf_packed_maps_bytes(L_r, d_r, d_in, dtype);
  const char* a0 = static_cast<const char*>(A);
  const char* p0 = static_cast<const char*>(A_packed);
  if (a0 < p0 + bytes && p0 < a0 + (bytes - HF_PACKED_HEADER_BYTES))
    return fail(HF_ERR_SHAPE, "A and A_packed overlap");
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  {
    TimedLaunch t(HF_KERNEL_PACK, s);
    e = hf::launch_pack_maps(dtype, 2 * L_r, d_r, d_in, A, A_packed, s);
  }
  if (e != hipSuccess) return hip_fail(e, "pack launch");
  return ok();
}

namespace {

struct RopeSizes {
  int P_s = 0, P_r = 0;  // table rows (0 = table not needed)
};

int32_t rope_sizes(int32_t B, const int32_t* s_len, const int32_t* r_len, const hf_rope* rope,
                   RopeSizes& rs) {
  rs = RopeSizes();
  if (!rope) return HF_OK;
  for (int b = 0; b < B; ++b) {
    const int64_t ps = rope->pos0_s ? rope->pos0_s[b] : 0;
    const int64_t pr = rope->pos0_r ? rope->pos0_r[b] : 0;
    if (ps < 0 || pr < 0) return fail(HF_ERR_SHAPE, "RoPE start positions must be >= 0");
    if (ps + s_len[b] > INT32_MAX || pr + r_len[b] > INT32_MAX)
      return fail(HF_ERR_SHAPE, "RoPE positions overflow int32");
    if (rope->unrotate_sender_k) rs.P_s = std::max(rs.P_s, (int)(ps + s_len[b]));
    if (rope->rotate_receiver_k) rs.P_r = std::max(rs.P_r, (int)(pr + r_len[b]));
  }
  // The bf16 kernels also read the rotations of the small offsets 0..15.
  if (rs.P_s > 0) rs.P_s = std::max(rs.P_s, hf::kRopeDeltaRows);
  return HF_OK;
}

size_t rope_bytes(int P, int d_h) { return align_up((size_t)P * d_h * sizeof(float), 256); }

// Staging records of the row tiles (one per tile of the batch) and the work
// counter after them, where the kernel that runs keeps them.
size_t record_bytes(int32_t B, const int32_t* r_len, const hf_kv_desc* sender,
                    const hf_kv_desc* receiver) {
  const size_t per = hf::transfer_tile_record_bytes(sender->dtype, receiver->H, sender->H,
                                                    sender->d_h);
  if (per == 0) return 0;
  const int rt = hf::transfer_rows_per_tile(sender->dtype, receiver->H, sender->H, 1, sender->d_h);
  size_t tiles = 0;
  for (int b = 0; b < B; ++b) tiles += r_len[b] > 0 ? ((size_t)r_len[b] + rt - 1) / rt : 0;
  return tiles * per + 256;
}

}  // namespace

namespace {

// Staged path: 256-row tiles of the batch and the workspace it adds to the
// fused path's (the RoPE table of positions 0..31, then the slabs).
int64_t staged_row_tiles(int32_t B, const int32_t* r_len) {
  int64_t n = 0;
  for (int b = 0; b < B; ++b) n += r_len[b] > 0 ? ((int64_t)r_len[b] + hf::kStagedRows - 1) / hf::kStagedRows : 0;
  return n;
}
size_t staged_extra_bytes(int32_t B, const int32_t* r_len, int n_slab_layers) {
  return hf::kStagedT1Bytes +
         (size_t)2 * n_slab_layers * (size_t)staged_row_tiles(B, r_len) * hf::kStagedRows * 1024 * 2;
}

}  // namespace

size_t hf_transfer_staged_workspace_bytes(int32_t B, const int32_t* s_len, const int32_t* r_len,
                                          const hf_kv_desc* sender, const hf_kv_desc* receiver,
                                          const hf_rope* rope, int32_t n_taps) {
  if (B < 1 || B > HF_MAX_BATCH || !s_len || !r_len || !sender || !receiver) return 0;
  if (n_taps < 0 || n_taps > 3) return 0;
  if (!hf::staged_supported(sender->dtype, sender->H, receiver->H, sender->d_h) ||
      receiver->d_h != sender->d_h)
    return 0;
  for (int b = 0; b < B; ++b)
    if (s_len[b] < 0 || r_len[b] < 0) return 0;
  const size_t base = hf_transfer_workspace_bytes(B, s_len, r_len, sender, receiver, rope);
  if (base == 0) return 0;
  return base + staged_extra_bytes(B, r_len, n_taps == 0 ? receiver->L : sender->L);
}

size_t hf_transfer_workspace_bytes(int32_t B, const int32_t* s_len, const int32_t* r_len,
                                   const hf_kv_desc* sender, const hf_kv_desc* receiver,
                                   const hf_rope* rope) {
  if (B < 1 || B > HF_MAX_BATCH || !s_len || !r_len || !sender || !receiver) return 0;
  RopeSizes rs;
  if (rope_sizes(B, s_len, r_len, rope, rs) != HF_OK) return 0;
  return rope_bytes(rs.P_s, sender->d_h) + rope_bytes(rs.P_r, receiver->d_h) +
         record_bytes(B, r_len, sender, receiver);
}

namespace {

// Which sender layers feed each receiver layer: an interpolation table
// (lo, hi, rem, den) or n_taps concatenated layers.
struct LayerSpec {
  bool concat = false;
  int32_t n_taps = 1;
  const int32_t* lo = nullptr;
  const int32_t* hi = nullptr;
  const int32_t* rem = nullptr;
  const int32_t* den_l = nullptr;
  const int32_t* taps = nullptr;  // [L_r][n_taps]
};

// timed: bracket the launches with profiler events (which create HIP events);
// the no-allocation entry point passes false.
int32_t transfer_impl(int32_t B, const int32_t* s_len, const int32_t* r_len,
                      const int32_t* row_ptr, const int32_t* col, const int32_t* num,
                      const int32_t* den, const LayerSpec& ls, const hf_kv_desc* sender,
                      const hf_kv_desc* receiver, const void* A_packed, size_t A_packed_bytes,
                      const float* bias, const hf_rope* rope, const hf_transfer_opts* opts,
                      void* workspace, size_t workspace_bytes, void* stream,
                      bool noalloc = false) {
  const bool timed = !noalloc;
  if (B < 1 || B > HF_MAX_BATCH) return fail(HF_ERR_SHAPE, "B=%d outside [1, %d]", B, HF_MAX_BATCH);
  if (!s_len || !r_len) return fail(HF_ERR_NULL, "s_len / r_len is NULL");
  if (ls.concat) {
    if (!ls.taps) return fail(HF_ERR_NULL, "layer taps table is NULL");
    if (ls.n_taps < 1 || ls.n_taps > 3) return fail(HF_ERR_SHAPE, "n_taps %d outside [1, 3]", ls.n_taps);
  } else if (!ls.lo || !ls.hi || !ls.rem || !ls.den_l) {
    return fail(HF_ERR_NULL, "layer table is NULL");
  }
  if (!row_ptr || !col || !num || !den) return fail(HF_ERR_NULL, "alignment table is NULL");
  if (!A_packed) return fail(HF_ERR_NULL, "A_packed is NULL");
  int32_t st;
  if ((st = check_desc("sender", sender)) || (st = check_desc("receiver", receiver))) return st;
  if (sender->dtype != receiver->dtype) return fail(HF_ERR_DTYPE, "sender and receiver dtypes differ");
  if (sender->d_h != receiver->d_h) return fail(HF_ERR_SHAPE, "sender and receiver d_h differ");
  const int dtype = sender->dtype, d_h = sender->d_h;
  const int L_s = sender->L, L_r = receiver->L;
  if (L_r > HF_MAX_LAYERS) return fail(HF_ERR_SHAPE, "receiver layers %d > %d", L_r, HF_MAX_LAYERS);
  if (L_s > 256) return fail(HF_ERR_SHAPE, "sender layers %d > 256", L_s);
  if (!aligned16(A_packed)) return fail(HF_ERR_SHAPE, "A_packed not 16-byte aligned");
  if (bias && (reinterpret_cast<uintptr_t>(bias) & 15u)) return fail(HF_ERR_SHAPE, "bias not 16-byte aligned");
  const int d_in = sender->H * d_h;   // one tap
  const int d_all = ls.n_taps * d_in;  // the map's input size
  {
    const size_t want = hf_packed_maps_bytes(L_r, receiver->H * d_h, d_all, dtype);
    if (A_packed_bytes != want)
      return fail(HF_ERR_SHAPE,
                  "A_packed holds %zu bytes, but maps packed by hf_pack_maps for L_r=%d, d_r=%d, "
                  "d_in=%d, dtype %d hold %zu (with their %d-byte header)", A_packed_bytes, L_r,
                  receiver->H * d_h, d_all, dtype, want, HF_PACKED_HEADER_BYTES);
  }
  if (dtype == HF_BF16) {
    if (d_h != 128) return fail(HF_ERR_UNSUPPORTED, "bf16 path needs d_h == 128 (got %d)", d_h);
    const int H = receiver->H;
    if (H != 2 && H != 4 && H != 8)
      return fail(HF_ERR_UNSUPPORTED, "bf16 path needs receiver H in {2,4,8} (got %d)", H);
    if ((int64_t)H * d_h * d_all * 2 >= ((int64_t)1 << 31))
      return fail(HF_ERR_UNSUPPORTED, "bf16 path needs one (layer, role) map under 2 GiB");
  } else if (d_all > 4096 || d_in % 4) {
    return fail(HF_ERR_UNSUPPORTED, "fp32 path needs n_taps*d_in <= 4096 and d_in %% 4 == 0");
  }
  int64_t sum_r = 0;
  for (int b = 0; b < B; ++b) {
    if (s_len[b] < 0 || r_len[b] < 0) return fail(HF_ERR_SHAPE, "negative length in sequence %d", b);
    if (s_len[b] > sender->T_cap || r_len[b] > receiver->T_cap)
      return fail(HF_ERR_SHAPE, "sequence %d longer than the cache capacity", b);
    if (r_len[b] > 0 && s_len[b] == 0)
      return fail(HF_ERR_SHAPE, "sequence %d has receiver tokens but no sender tokens", b);
    sum_r += r_len[b];
  }
  if (sum_r > INT32_MAX) return fail(HF_ERR_SHAPE, "too many receiver tokens");
  for (int j = 0; j < L_r; ++j) {
    if (ls.concat) {
      for (int t = 0; t < ls.n_taps; ++t) {
        const int32_t v = ls.taps[(int64_t)j * ls.n_taps + t];
        if (v < 0 || v >= L_s)
          return fail(HF_ERR_SHAPE, "taps row %d names a sender layer outside [0, %d)", j, L_s);
      }
      continue;
    }
    if (ls.lo[j] < 0 || ls.lo[j] >= L_s || ls.hi[j] < 0 || ls.hi[j] >= L_s)
      return fail(HF_ERR_SHAPE, "layer table row %d names a sender layer outside [0, %d)", j, L_s);
    if (ls.den_l[j] < 1 || ls.rem[j] < 0 || ls.rem[j] >= ls.den_l[j])
      return fail(HF_ERR_SHAPE, "layer table row %d needs 0 <= rem < den", j);
  }
  if (rope && (!(rope->theta_s > 0) || !(rope->theta_r > 0) || !std::isfinite(rope->theta_s) ||
               !std::isfinite(rope->theta_r)))
    return fail(HF_ERR_SHAPE, "RoPE thetas must be finite and > 0");
  if (opts) {
    if ((opts->inv_r && (reinterpret_cast<uintptr_t>(opts->inv_r) & 3u)) ||
        (opts->k_norm && (reinterpret_cast<uintptr_t>(opts->k_norm) & 3u)))
      return fail(HF_ERR_SHAPE, "opts buffers must be 4-byte aligned");
    if (opts->k_norm && !(std::isfinite(opts->k_norm_eps) && opts->k_norm_eps >= 0.0f))
      return fail(HF_ERR_SHAPE, "k_norm_eps must be finite and >= 0");
    if (opts->k_norm && dtype == HF_F32 && d_h != 64 && d_h != 128)
      return fail(HF_ERR_UNSUPPORTED, "fp32 key normalization needs d_h in {64, 128}");
  }
  RopeSizes rs;
  if ((st = rope_sizes(B, s_len, r_len, rope, rs))) return st;
  const size_t rec_off = rope_bytes(rs.P_s, d_h) + rope_bytes(rs.P_r, d_h);
  const size_t ws_need = rec_off + record_bytes(B, r_len, sender, receiver);
  if (noalloc && ws_need > HF_NOALLOC_SCRATCH_BYTES)
    return fail(HF_ERR_CAPACITY,
                "this transfer needs %zu bytes of scratch, more than the %d bytes "
                "hf_transfer_kv_noalloc holds; use hf_transfer_kv with a workspace",
                ws_need, HF_NOALLOC_SCRATCH_BYTES);
  // The staged path, where it applies and the workspace holds its slabs.
  bool staged = false;
  size_t st_need = 0;
  if (!noalloc && hf::staged_supported(dtype, sender->H, receiver->H, d_h) && ws_need > 0) {
    st_need = ws_need + staged_extra_bytes(B, r_len, ls.concat ? L_s : L_r);
    staged = workspace_bytes >= st_need;
    for (int b = 0; staged && b < B; ++b)  // receiver rows are addressed with 32-bit byte offsets
      if ((int64_t)r_len[b] * receiver->stride_t * 2 + 256 >= ((int64_t)1 << 31)) staged = false;
  }
  if (ws_need > 0 && !noalloc) {
    if (!workspace) return fail(HF_ERR_NULL, "workspace is NULL");
    if (workspace_bytes < ws_need)
      return fail(HF_ERR_CAPACITY, "workspace %zu bytes < required %zu", workspace_bytes, ws_need);
    if (reinterpret_cast<uintptr_t>(workspace) & 255u)
      return fail(HF_ERR_SHAPE, "workspace is not 256-byte aligned");
  }

  hf::TransferArgs a;
  std::memset(&a, 0, sizeof a);
  a.S = sender->ptr;
  a.R = receiver->ptr;
  a.Wp = static_cast<const char*>(A_packed) + HF_PACKED_HEADER_BYTES;
  a.bias = bias;
  if (opts) {
    a.inv_r = opts->inv_r;
    a.k_norm = opts->k_norm;
    a.k_norm_eps = opts->k_norm_eps;
  }
  a.row_ptr = row_ptr;
  a.col = col;
  a.num = num;
  a.den = den;
  a.s_sb = sender->stride_b; a.s_sl = sender->stride_l; a.s_sc = sender->stride_c;
  a.s_sh = sender->stride_h; a.s_st = sender->stride_t;
  a.r_sb = receiver->stride_b; a.r_sl = receiver->stride_l; a.r_sc = receiver->stride_c;
  a.r_sh = receiver->stride_h; a.r_st = receiver->stride_t;
  a.L_r = L_r;
  a.H_s = sender->H;
  a.H_r = receiver->H;
  a.d_h = d_h;
  a.B = B;
  a.n_taps = ls.n_taps;
  a.concat = ls.concat ? 1 : 0;
  a.rows_per_tile = hf::transfer_rows_per_tile(dtype, receiver->H, sender->H, ls.n_taps, d_h);
  int tiles = 0, row0 = 0;
  for (int b = 0; b < B; ++b) {
    a.tile_start[b] = tiles;
    tiles += (r_len[b] + a.rows_per_tile - 1) / a.rows_per_tile;
    a.Ts[b] = s_len[b];
    a.Tr[b] = r_len[b];
    a.row0[b] = row0;
    row0 += r_len[b];
    a.pos0_s[b] = rope && rope->pos0_s ? rope->pos0_s[b] : 0;
    a.pos0_r[b] = rope && rope->pos0_r ? rope->pos0_r[b] : 0;
  }
  a.tile_start[B] = tiles;
  {  // bytes one (sequence, layer, role) slab of the sender cache spans
    int Tmax = 1;
    for (int b = 0; b < B; ++b) Tmax = std::max(Tmax, (int)s_len[b]);
    const int64_t ext = ((int64_t)(sender->H - 1) * sender->stride_h +
                         (int64_t)(Tmax - 1) * sender->stride_t + d_h) * (dtype == HF_BF16 ? 2 : 4);
    a.s_extent = ext < ((int64_t)1 << 31) - 4096 ? (int32_t)ext : 0;
  }
  a.tiles_per_lc = tiles;
  if ((int64_t)tiles * L_r * 2 > INT32_MAX) return fail(HF_ERR_SHAPE, "too many work items");
  for (int j = 0; j < L_r; ++j) {
    if (ls.concat) {  // each tap is one sender layer with weight 1
      for (int t = 0; t < ls.n_taps; ++t) a.taps[j][t] = (uint8_t)ls.taps[(int64_t)j * ls.n_taps + t];
      a.lo[j] = a.hi[j] = a.taps[j][0];
      a.wlo[j] = 1.0f;
      a.whi[j] = 0.0f;
      continue;
    }
    a.lo[j] = (uint8_t)ls.lo[j];
    a.hi[j] = (uint8_t)ls.hi[j];
    a.taps[j][0] = a.lo[j];
    a.wlo[j] = (float)((double)(ls.den_l[j] - ls.rem[j]) / (double)ls.den_l[j]);
    a.whi[j] = (float)((double)ls.rem[j] / (double)ls.den_l[j]);
  }
  if (noalloc && ws_need > 0) {  // every host check has passed: the library's scratch array
    workspace = nullptr;
    const hipError_t se = hf::noalloc_scratch(&workspace);
    if (se != hipSuccess) return hip_fail(se, "scratch symbol address");
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(workspace);
  if (rope && rope->unrotate_sender_k && rs.P_s > 0) {
    a.cs_s = reinterpret_cast<const float*>(w);
    a.unrot = 1;
  }
  if (rope && rope->rotate_receiver_k && rs.P_r > 0) {
    a.cs_r = reinterpret_cast<const float*>(w + rope_bytes(rs.P_s, d_h));
    a.rot = 1;
  }
  if (ws_need > rec_off) {
    a.tile_rec = reinterpret_cast<const int32_t*>(w + rec_off);
    a.work_ctr = reinterpret_cast<int32_t*>(w + ws_need - 256);
  }
  if (staged) {
    a.cs_t1 = reinterpret_cast<const float*>(w + ws_need);
    a.xs = reinterpret_cast<uint16_t*>(w + ws_need + hf::kStagedT1Bytes);
    a.n_slab_layers = ls.concat ? L_s : L_r;
    int rt = 0;
    for (int b = 0; b < B; ++b) {
      a.rt_start[b] = rt;
      rt += (r_len[b] + hf::kStagedRows - 1) / hf::kStagedRows;
    }
    a.rt_start[B] = rt;
    a.n_rt = rt;
    a.xs_slab = (long long)rt * hf::kStagedRows * 1024;
  }
  if (tiles == 0) return ok();
  if (a.tile_rec) {
    int dev = 0, n_cu = 0;
    hipError_t de = hipGetDevice(&dev);
    if (de == hipSuccess) de = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
    if (de != hipSuccess) return hip_fail(de, "device query");
    a.n_wg = hf::transfer_persistent_grid(a, n_cu > 0 ? n_cu : 1);
  }
  hipError_t e = hipSuccess;
  if (a.unrot || a.rot) {
    TimedLaunch t(HF_KERNEL_ROPE_TABLES, s, timed);
    if (a.unrot) e = hf::launch_rope_table(const_cast<float*>(a.cs_s), rs.P_s, d_h, rope->theta_s, s);
    if (e == hipSuccess && a.rot)
      e = hf::launch_rope_table(const_cast<float*>(a.cs_r), rs.P_r, d_h, rope->theta_r, s);
    if (e == hipSuccess && a.rot && staged)  // positions 0..31 for the staged epilogue
      e = hf::launch_rope_table(const_cast<float*>(a.cs_t1), 32, d_h, rope->theta_r, s);
  }
  if (e != hipSuccess) return hip_fail(e, "RoPE table launch");
  if (a.tile_rec) {
    TimedLaunch t(HF_KERNEL_TRANSFER_STAGE, s, timed);
    e = hf::launch_transfer_stage(dtype, a, s);
  }
  if (e != hipSuccess) return hip_fail(e, "tile staging launch");
  if (staged) {
    {
      TimedLaunch t(HF_KERNEL_STAGED_BUILD, s, timed);
      e = hf::launch_staged_build(a, s);
    }
    if (e != hipSuccess) return hip_fail(e, "staged build launch");
    {
      TimedLaunch t(HF_KERNEL_STAGED_GEMM, s, timed);
      e = hf::launch_staged_gemm(a, s);
    }
    if (e != hipSuccess) return hip_fail(e, "staged multiply launch");
    return ok();
  }
  {
    TimedLaunch t(HF_KERNEL_TRANSFER, s, timed);
    e = hf::launch_transfer(dtype, a, s);
  }
  if (e != hipSuccess) return hip_fail(e, "transfer launch");
  return ok();
}

}  // namespace

int32_t hf_transfer_kv(int32_t B, const int32_t* s_len, const int32_t* r_len,
                       const int32_t* row_ptr, const int32_t* col, const int32_t* num,
                       const int32_t* den, const int32_t* lo, const int32_t* hi,
                       const int32_t* rem, const int32_t* den_l, const hf_kv_desc* sender,
                       const hf_kv_desc* receiver, const void* A_packed, size_t A_packed_bytes,
                       const float* bias, const hf_rope* rope, const hf_transfer_opts* opts,
                       void* workspace, size_t workspace_bytes, void* stream) {
  LayerSpec ls;
  ls.lo = lo;
  ls.hi = hi;
  ls.rem = rem;
  ls.den_l = den_l;
  return transfer_impl(B, s_len, r_len, row_ptr, col, num, den, ls, sender, receiver, A_packed,
                       A_packed_bytes, bias, rope, opts, workspace, workspace_bytes, stream);
}

int32_t hf_transfer_kv_noalloc(int32_t B, const int32_t* s_len, const int32_t* r_len,
                               const int32_t* row_ptr, const int32_t* col, const int32_t* num,
                               const int32_t* den, const int32_t* lo, const int32_t* hi,
                               const int32_t* rem, const int32_t* den_l,
                               const hf_kv_desc* sender, const hf_kv_desc* receiver,
                               const void* A_packed, size_t A_packed_bytes, const float* bias,
                               const hf_rope* rope, const hf_transfer_opts* opts, void* stream) {
  LayerSpec ls;
  ls.lo = lo;
  ls.hi = hi;
  ls.rem = rem;
  ls.den_l = den_l;
  return transfer_impl(B, s_len, r_len, row_ptr, col, num, den, ls, sender, receiver, A_packed,
                       A_packed_bytes, bias, rope, opts, nullptr, 0, stream, /*noalloc=*/true);
}

int32_t hf_transfer_kv_taps(int32_t B, const int32_t* s_len, const int32_t* r_len,
                            const int32_t* row_ptr, const int32_t* col, const int32_t* num,
                            const int32_t* den, int32_t n_taps, const int32_t* taps,
                            const hf_kv_desc* sender, const hf_kv_desc* receiver,
                            const void* A_packed, size_t A_packed_bytes, const float* bias,
                            const hf_rope* rope, const hf_transfer_opts* opts, void* workspace,
                            size_t workspace_bytes, void* stream) {
  LayerSpec ls;
  ls.concat = true;
  ls.n_taps = n_taps;
  ls.taps = taps;
  return transfer_impl(B, s_len, r_len, row_ptr, col, num, den, ls, sender, receiver, A_packed,
                       A_packed_bytes, bias, rope, opts, workspace, workspace_bytes, stream);
}

// ---------------------------------------------------------------------------
// Offline map construction.
// ---------------------------------------------------------------------------

size_t hf_recolor_moments_workspace_bytes(int64_t n, int32_t p, int32_t q) {
  if (n < 1 || p < 1 || q < 1) return 0;
  return hf::recolor_moments_workspace_bytes(n, p, q);
}

size_t hf_recolor_solve_workspace_bytes(int32_t p, int32_t q) {
  if (p < 1 || q < 1) return 0;
  return hf::recolor_solve_workspace_bytes(p, q);
}

size_t hf_fold_workspace_bytes(int32_t p, int32_t rank) {
  if (p < 1 || rank < 1) return 0;
  return hf::fold_workspace_bytes(p, rank);
}

namespace {

constexpr int32_t kMaxFeatures = 65536;
constexpr int64_t kMaxGemmRows = 65535LL * 64;  // row tiles of 64 on the grid's y axis

bool aligned_to(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  const char* x = static_cast<const char*>(a);
  const char* y = static_cast<const char*>(b);
  return x < y + nb && y < x + na;
}

int32_t check_workspace(const void* ws, size_t bytes, size_t need) {
  if (!ws) return fail(HF_ERR_NULL, "workspace is NULL");
  if (!aligned_to(ws, 256)) return fail(HF_ERR_SHAPE, "workspace is not 256-byte aligned");
  if (bytes < need) return fail(HF_ERR_CAPACITY, "workspace %zu bytes < required %zu", bytes, need);
  return HF_OK;
}

}  // namespace

int32_t hf_recolor_moments(int64_t n, int32_t p, int32_t q, int32_t dtype, const void* x,
                           int64_t ldx, const void* y, int64_t ldy, const float* w, double* r,
                           double* mu, double* cov, void* workspace, size_t workspace_bytes,
                           void* stream) {
  if (n < 1) return fail(HF_ERR_SHAPE, "need n >= 1 samples");
  if (p < 1 || q < 1 || p > kMaxFeatures || q > kMaxFeatures || p + q > kMaxFeatures)
    return fail(HF_ERR_SHAPE, "need p, q >= 1 and p + q <= %d", kMaxFeatures);
  if (dtype != HF_F32 && dtype != HF_BF16) return fail(HF_ERR_DTYPE, "dtype %d unknown", dtype);
  if (!x || !y || !r || !mu || !cov) return fail(HF_ERR_NULL, "x / y / r / mu / cov is NULL");
  if (ldx < p || ldy < q) return fail(HF_ERR_SHAPE, "need ldx >= p and ldy >= q");
  const size_t es = dtype == HF_BF16 ? 2 : 4;
  if (!aligned_to(x, es) || !aligned_to(y, es) || (w && !aligned_to(w, 4)))
    return fail(HF_ERR_SHAPE, "x / y / w not aligned to their element size");
  if (!aligned_to(r, 8) || !aligned_to(mu, 8) || !aligned_to(cov, 8))
    return fail(HF_ERR_SHAPE, "r / mu / cov not 8-byte aligned");
  const size_t pq = (size_t)p + q;
  if (overlap(cov, pq * pq * 8, mu, pq * 8) || overlap(cov, pq * pq * 8, r, 8) ||
      overlap(mu, pq * 8, r, 8))
    return fail(HF_ERR_SHAPE, "r, mu and cov overlap");
  int32_t st;
  if ((st = check_workspace(workspace, workspace_bytes, hf::recolor_moments_workspace_bytes(n, p, q))))
    return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  {
    TimedLaunch t(HF_KERNEL_MOMENTS_STATS, s);
    e = hf::launch_recolor_stats(dtype, n, p, q, x, ldx, y, ldy, w, r, mu, workspace, s);
  }
  if (e != hipSuccess) return hip_fail(e, "moments statistics launch");
  {
    TimedLaunch t(HF_KERNEL_MOMENTS_COV, s);
    e = hf::launch_recolor_cov(dtype, n, p, q, x, ldx, y, ldy, w, workspace, s);
  }
  if (e != hipSuccess) return hip_fail(e, "covariance launch");
  {
    TimedLaunch t(HF_KERNEL_MOMENTS_STATS, s);
    e = hf::launch_recolor_cov_reduce(n, p, q, cov, workspace, s);
  }
  if (e != hipSuccess) return hip_fail(e, "covariance reduction launch");
  return ok();
}

int32_t hf_recolor_solve(int32_t p, int32_t q, const double* mu, const double* cov, double ridge,
                         double* A, double* b, hf_recolor_info* info, void* workspace,
                         size_t workspace_bytes, void* stream) {
  if (p < 1 || q < 1 || p > kMaxFeatures || q > kMaxFeatures || p + q > kMaxFeatures)
    return fail(HF_ERR_SHAPE, "need p, q >= 1 and p + q <= %d", kMaxFeatures);
  if (!(ridge >= 0.0) || !std::isfinite(ridge)) return fail(HF_ERR_SHAPE, "ridge must be finite and >= 0");
  if (!mu || !cov || !A || !b) return fail(HF_ERR_NULL, "mu / cov / A / b is NULL");
  if (!aligned_to(mu, 8) || !aligned_to(cov, 8) || !aligned_to(A, 8) || !aligned_to(b, 8) ||
      (info && !aligned_to(info, 8)))
    return fail(HF_ERR_SHAPE, "mu / cov / A / b / info not 8-byte aligned");
  const size_t pq = (size_t)p + q, nA = (size_t)p * q * 8, nb = (size_t)q * 8;
  if (overlap(A, nA, b, nb) || overlap(A, nA, mu, pq * 8) || overlap(A, nA, cov, pq * pq * 8) ||
      overlap(b, nb, mu, pq * 8) || overlap(b, nb, cov, pq * pq * 8))
    return fail(HF_ERR_SHAPE, "outputs A / b overlap each other or the inputs");
  int32_t st;
  if ((st = check_workspace(workspace, workspace_bytes, hf::recolor_solve_workspace_bytes(p, q))))
    return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  {
    TimedLaunch t(HF_KERNEL_RECOLOR_SOLVE, s);
    e = hf::launch_recolor_solve(p, q, mu, cov, ridge, A, b, info, workspace, s);
  }
  if (e != hipSuccess) return hip_fail(e, "recolor launch");
  return ok();
}

int32_t hf_fold_map(int32_t p, int32_t q, int32_t rank, const double* A, const double* b,
                    const double* B, const double* G, double* A_out, double* b_out,
                    void* workspace, size_t workspace_bytes, void* stream) {
  if (p < 1 || q < 1 || rank < 1 || p > kMaxFeatures || q > kMaxFeatures || rank > kMaxFeatures)
    return fail(HF_ERR_SHAPE, "need 1 <= p, q, rank <= %d", kMaxFeatures);
  if (!A || !b || !B || !G || !A_out || !b_out) return fail(HF_ERR_NULL, "an argument is NULL");
  const void* ptrs[6] = {A, b, B, G, A_out, b_out};
  for (const void* ptr : ptrs)
    if (!aligned_to(ptr, 8)) return fail(HF_ERR_SHAPE, "pointers must be 8-byte aligned");
  const size_t nA = (size_t)p * q * 8, nb = (size_t)q * 8, nB = (size_t)q * rank * 8;
  if ((A_out != A && overlap(A_out, nA, A, nA)) || (b_out != b && overlap(b_out, nb, b, nb)))
    return fail(HF_ERR_SHAPE, "A_out / b_out must be A / b exactly or not overlap them");
  if (overlap(A_out, nA, b_out, nb) || overlap(A_out, nA, B, nB) || overlap(A_out, nA, G, nB) ||
      overlap(b_out, nb, B, nB) || overlap(b_out, nb, G, nB) || overlap(A_out, nA, b, nb) ||
      overlap(b_out, nb, A, nA))
    return fail(HF_ERR_SHAPE, "outputs overlap other arguments");
  int32_t st;
  if ((st = check_workspace(workspace, workspace_bytes, hf::fold_workspace_bytes(p, rank)))) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  {
    TimedLaunch t(HF_KERNEL_FOLD, s);
    e = hf::launch_fold(p, q, rank, A, b, B, G, A_out, b_out, workspace, s);
  }
  if (e != hipSuccess) return hip_fail(e, "fold launch");
  return ok();
}

int32_t hf_gemm_f64(int32_t m, int32_t n, int64_t k, const double* A, int64_t lda,
                    int32_t a_kmajor, const double* B, int64_t ldb, int32_t b_kmajor, double* D,
                    int64_t ldd, double alpha, double beta, const double* C, int64_t ldc,
                    double gamma, void* stream) {
  if (m < 1 || n < 1 || k < 0 || m > kMaxGemmRows)
    return fail(HF_ERR_SHAPE, "need 1 <= m <= %lld, n >= 1, k >= 0", (long long)kMaxGemmRows);
  if (!D || (k > 0 && (!A || !B))) return fail(HF_ERR_NULL, "A / B / D is NULL");
  if (beta != 0.0 && !C) return fail(HF_ERR_NULL, "C is NULL with beta != 0");
  if (k > 0 && (lda < (a_kmajor ? m : k) || ldb < (b_kmajor ? n : k)))
    return fail(HF_ERR_SHAPE, "lda / ldb too small for the layouts");
  if (ldd < n || (beta != 0.0 && ldc < n)) return fail(HF_ERR_SHAPE, "ldd / ldc < n");
  if (!aligned_to(D, 8) || (A && !aligned_to(A, 8)) || (B && !aligned_to(B, 8)) ||
      (C && !aligned_to(C, 8)))
    return fail(HF_ERR_SHAPE, "pointers must be 8-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const hipError_t e = hf::launch_gemm_f64(m, n, k, A, lda, a_kmajor, B, ldb, b_kmajor, D, ldd,
                                           alpha, beta, C, ldc, gamma, s);
  if (e != hipSuccess) return hip_fail(e, "gemm launch");
  return ok();
}

int32_t hf_profiler_enable(int32_t on) {
  Profiler& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  p.on = on != 0;
  return ok();
}

int32_t hf_profiler_reset(void) {
  Profiler& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  int32_t st = drain_profiler(p);
  for (int k = 0; k < HF_KERNEL_COUNT; ++k) {
    p.total_ms[k] = 0.0;
    p.launches[k] = 0;
    p.samples[k].clear();
  }
  return st == HF_OK ? ok() : st;
}

int32_t hf_profiler_query(int32_t kernel_id, double* total_ms, int64_t* launches) {
  if (kernel_id < 0 || kernel_id >= HF_KERNEL_COUNT) return fail(HF_ERR_SHAPE, "kernel id %d unknown", kernel_id);
  if (!total_ms || !launches) return fail(HF_ERR_NULL, "output pointer is NULL");
  Profiler& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  int32_t st = drain_profiler(p);
  if (st != HF_OK) return st;
  *total_ms = p.total_ms[kernel_id];
  *launches = p.launches[kernel_id];
  return ok();
}

int32_t hf_profiler_samples(int32_t kernel_id, float* ms, int64_t capacity, int64_t* count) {
  if (kernel_id < 0 || kernel_id >= HF_KERNEL_COUNT) return fail(HF_ERR_SHAPE, "kernel id %d unknown", kernel_id);
  if (!count || (capacity > 0 && !ms)) return fail(HF_ERR_NULL, "output pointer is NULL");
  Profiler& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  const int32_t st = drain_profiler(p);
  if (st != HF_OK) return st;
  const std::vector<float>& v = p.samples[kernel_id];
  const int64_t n = std::min<int64_t>(capacity, (int64_t)v.size());
  for (int64_t k = 0; k < n; ++k) ms[k] = v[k];
  *count = (int64_t)v.size();
  return ok();
}

}  // extern "C"
