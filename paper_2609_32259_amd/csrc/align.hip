// Cross-tokenizer alignment kernels (Sec. 3.1 "Token Alignment"; App. B.1),
// producing the CSR span table described in heterofold.h.
//
// Integer-only, three launches:
//   1. align_count: per receiver token, binary searches over the sender
//      spans give the TA partner (sender token ending at the same character)
//      and the number of overlapping sender tokens.  Per-workgroup totals go
//      to the workspace.  The counts and partners are parked in row_ptr / den.
//   2. align_scan: one workgroup scans the per-workgroup totals (entry
//      offsets) and the per-workgroup last partners (forward fill carried
//      across workgroups of the same sequence), and finds each sequence's
//      first nonempty sender token.
//   3. align_fill: per receiver token, the final offsets and forward-filled
//      partner, then the entries themselves.
// Each receiver row is handled by the same thread in launches 1 and 3, and
// rows' parked values live in their own slots, so no launch reads another
// workgroup's parked data.
#include <hip/hip_runtime.h>
#include <limits.h>

#include "hf_internal.h"

namespace hf {
namespace {

constexpr int kScanThreads = 1024;

__device__ __forceinline__ int upper_bound_dev(const int32_t* a, int n, int x) {
  int lo = 0, hi = n;  // first index with a[i] > x
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if (a[mid] > x) hi = mid; else lo = mid + 1;
  }
  return lo;
}

__device__ __forceinline__ int lower_bound_dev(const int32_t* a, int n, int x) {
  int lo = 0, hi = n;  // first index with a[i] >= x
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if (a[mid] >= x) hi = mid; else lo = mid + 1;
  }
  return lo;
}

struct Plus {
  __device__ long long operator()(long long a, long long b) const { return a + b; }
};
struct LastValid {  // keeps the right operand unless it is "none" (negative)
  __device__ long long operator()(long long a, long long b) const { return b >= 0 ? b : a; }
};
struct Min {
  __device__ long long operator()(long long a, long long b) const { return b < a ? b : a; }
};

template <typename Op>
__device__ __forceinline__ long long wave_inclusive_scan(long long v, Op op) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    long long o = __shfl_up(v, d, 64);
    if (lane >= d) v = op(o, v);
  }
  return v;
}

// Inclusive scan over the workgroup (threads in order); also returns the
// workgroup total.  smem: NT/64 entries.  All threads must call it.
template <int NT, typename Op>
__device__ long long block_inclusive_scan(long long v, Op op, long long identity,
                                          long long* smem, long long& total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  v = wave_inclusive_scan(v, op);
  if (lane == 63) smem[wid] = v;
  __syncthreads();
  long long prefix = identity, tot = identity;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) {
    if (w < wid) prefix = op(prefix, smem[w]);
    tot = op(tot, smem[w]);
  }
  __syncthreads();
  total = tot;
  return op(prefix, v);
}

__device__ __forceinline__ int seq_of_block(const AlignArgs& p, int blk) {
  int b = 0;
  while (b + 1 < p.B && p.blk_start[b + 1] <= blk) ++b;
  return b;
}

// TA partner of receiver token j (or -1) and, in overlap mode, the number of
// sender tokens sharing at least one character with it (0 if none).
struct RowInfo {
  int partner;
  int count;
  int lo, hi;  // overlap candidate range [lo, hi)
};

__device__ __forceinline__ RowInfo row_info(const AlignArgs& p, const int32_t* sb,
                                            const int32_t* se, int Ts, int rb, int re) {
  RowInfo r;
  r.partner = -1;
  if (rb < re) {
    int i = upper_bound_dev(se, Ts, re) - 1;  // last sender token ending at or before re
    while (i >= 0 && se[i] == re && !(sb[i] < se[i])) --i;  // skip empty tokens at re
    if (i >= 0 && se[i] == re && sb[i] < se[i]) r.partner = i;
  }
  r.count = 1;
  r.lo = r.hi = 0;
  if (p.mode == HF_ALIGN_OVERLAP) {
    r.lo = upper_bound_dev(se, Ts, rb);  // first sender token ending after rb
    r.hi = lower_bound_dev(sb, Ts, re);  // first sender token starting at or after re
    int c = 0;
    for (int i = r.lo; i < r.hi; ++i) {
      int o = min(se[i], re) - max(sb[i], rb);
      c += (o > 0);
    }
    r.count = c;
  }
  return r;
}

__global__ __launch_bounds__(kAlignBlock) void align_count_kernel(const AlignArgs p) {
  __shared__ long long red[kAlignBlock / 64];
  const int blk = blockIdx.x;
  const int b = seq_of_block(p, blk);
  const int j = (blk - p.blk_start[b]) * kAlignBlock + threadIdx.x;
  const bool valid = j < p.Tr[b];
  const int32_t* sb = p.s_beg + p.s0[b];
  const int32_t* se = p.s_end + p.s0[b];
  long long cnt = 0, part = -1;
  if (valid) {
    const int g = p.r0[b] + j;
    RowInfo r = row_info(p, sb, se, p.Ts[b], p.r_beg[g], p.r_end[g]);
    int c = (p.mode == HF_ALIGN_OVERLAP) ? (r.count > 0 ? r.count : 1) : 1;
    p.row_ptr[g] = c;          // parked: entry count of row g
    p.den[g] = r.partner;      // parked: TA partner of row g
    cnt = c;
    part = r.partner;
  }
  long long tot_cnt, tot_part;
  block_inclusive_scan<kAlignBlock>(cnt, Plus(), 0, red, tot_cnt);
  block_inclusive_scan<kAlignBlock>(part, LastValid(), -1, red, tot_part);
  if (threadIdx.x == 0) {
    p.blk_sum[blk] = tot_cnt;
    p.blk_last[blk] = (int32_t)tot_part;
  }
}

__global__ __launch_bounds__(kScanThreads) void align_scan_kernel(const AlignArgs p) {
  __shared__ long long red[kScanThreads / 64];
  __shared__ long long incl_last[kScanThreads];
  __shared__ int first_ne[HF_MAX_BATCH];
  const int tid = threadIdx.x;

  // First nonempty sender token of each sequence (0 if there is none).
  for (int b = 0; b < p.B; ++b) {
    long long found = LLONG_MAX;
    for (int base = 0; base < p.Ts[b]; base += kScanThreads) {
      int i = base + tid;
      long long cand = LLONG_MAX;
      if (i < p.Ts[b] && p.s_beg[p.s0[b] + i] < p.s_end[p.s0[b] + i]) cand = i;
      long long m;
      block_inclusive_scan<kScanThreads>(cand, Min(), LLONG_MAX, red, m);
      if (m != LLONG_MAX) {
        found = m;
        break;
      }
    }
    if (tid == 0) first_ne[b] = (found == LLONG_MAX) ? 0 : (int)found;
  }
  __syncthreads();

  long long sum_carry = 0, last_carry = -1;
  for (int base = 0; base < p.nblk; base += kScanThreads) {
    const int k = base + tid;
    const bool valid = k < p.nblk;
    const int bs = valid ? seq_of_block(p, k) : 0;
    long long s = valid ? p.blk_sum[k] : 0;
    // Tag partners with their sequence so a carry never crosses sequences.
    long long lv = (valid && p.blk_last[k] >= 0) ? (((long long)bs << 32) | p.blk_last[k]) : -1;
    long long tot_s, tot_l;
    long long incl_s = block_inclusive_scan<kScanThreads>(s, Plus(), 0, red, tot_s);
    long long incl_l = block_inclusive_scan<kScanThreads>(lv, LastValid(), -1, red, tot_l);
    incl_last[tid] = incl_l;
    __syncthreads();
    if (valid) {
      p.blk_off[k] = sum_carry + incl_s - s;
      long long before = tid > 0 ? LastValid()(last_carry, incl_last[tid - 1]) : last_carry;
      p.blk_carry[k] = (before >= 0 && (before >> 32) == bs) ? (int32_t)(before & 0xffffffffLL)
                                                             : first_ne[bs];
    }
    sum_carry += tot_s;
    last_carry = LastValid()(last_carry, tot_l);
    __syncthreads();
  }
  if (tid == 0) p.row_ptr[p.total_rows] = (int32_t)(sum_carry < p.cap ? sum_carry : p.cap);
}

__global__ __launch_bounds__(kAlignBlock) void align_fill_kernel(const AlignArgs p) {
  __shared__ long long red[kAlignBlock / 64];
  const int blk = blockIdx.x;
  const int b = seq_of_block(p, blk);
  const int j = (blk - p.blk_start[b]) * kAlignBlock + threadIdx.x;
  const bool valid = j < p.Tr[b];
  const int g = p.r0[b] + j;
  long long cnt = valid ? p.row_ptr[g] : 0;
  long long part = valid ? p.den[g] : -1;
  long long tot;
  long long off = block_inclusive_scan<kAlignBlock>(cnt, Plus(), 0, red, tot) - cnt + p.blk_off[blk];
  long long fill = block_inclusive_scan<kAlignBlock>(part, LastValid(), -1, red, tot);
  if (!valid) return;
  const int a = fill >= 0 ? (int)fill : p.blk_carry[blk];
  p.row_ptr[g] = (int32_t)(off < p.cap ? off : p.cap);
  if (p.mode == HF_ALIGN_TA) {
    if (off < p.cap) {
      p.col[off] = a;
      p.num[off] = 1;
    }
    p.den[g] = 1;
    return;
  }
  const int32_t* sb = p.s_beg + p.s0[b];
  const int32_t* se = p.s_end + p.s0[b];
  const int rb = p.r_beg[g], re = p.r_end[g];
  RowInfo r = row_info(p, sb, se, p.Ts[b], rb, re);
  if (r.count == 0) {
    if (off < p.cap) {
      p.col[off] = a;
      p.num[off] = 1;
    }
    p.den[g] = 1;
    return;
  }
  int total = 0;
  long long e = off;
  for (int i = r.lo; i < r.hi; ++i) {
    int o = min(se[i], re) - max(sb[i], rb);
    if (o > 0) {
      if (e < p.cap) {
        p.col[e] = i;
        p.num[e] = o;
      }
      ++e;
      total += o;
    }
  }
  p.den[g] = total;
}

}  // namespace

size_t align_workspace_bytes(int nblk) {
  size_t n = (size_t)(nblk > 0 ? nblk : 1);
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  return 2 * up(n * sizeof(long long)) + 2 * up(n * sizeof(int32_t));
}

hipError_t launch_alignment(const AlignArgs& a, hipStream_t s) {
  if (a.nblk > 0) {
    hipLaunchKernelGGL(align_count_kernel, dim3(a.nblk), dim3(kAlignBlock), 0, s, a);
  }
  hipLaunchKernelGGL(align_scan_kernel, dim3(1), dim3(kScanThreads), 0, s, a);
  if (a.nblk > 0) {
    hipLaunchKernelGGL(align_fill_kernel, dim3(a.nblk), dim3(kAlignBlock), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace hf
