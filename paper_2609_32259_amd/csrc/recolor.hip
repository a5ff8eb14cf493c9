// Offline construction of the folded affine maps on the GPU, in fp64:
//   * weighted sender RMS (Eq. 3), means and the joint covariance of [x/r | y]
//     (Sec. 3.2) -- one weighted, centred Gram product over all samples;
//   * Recolor (Eq. 4-5): symmetric roots of the covariances and the Procrustes
//     factor R* = U Q^T of the whitened cross-covariance, by Newton-Schulz
//     iterations (matrix products only; R* is the polar factor of that matrix);
//   * the fold of the low-rank correction into the map (Eq. 9).
//
// Every product runs on one fp64 matrix-core GEMM kernel
// (v_mfma_f64_16x16x4f64).  The iterations run without host synchronization:
// a small state record in device memory tells the remaining launches of a
// converged iteration to do nothing.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "hf_internal.h"

namespace hf {
namespace {

typedef double double4_t __attribute__((ext_vector_type(4)));

constexpr int kBM = 64, kBN = 64, kBK = 16, kPad = 4;
constexpr int kGemmThreads = 256;
constexpr int kRedThreads = 256;
constexpr int kMaxRedBlocks = 1024;

// Newton-Schulz convergence: once the residual |I - P|_F falls below this, the
// error contracts as e' = 3/4 e^2 + e^3/4, so three more steps reach rounding.
constexpr double kNsSwitch = 1e-3;
constexpr int kNsExtra = 2;

struct NsState {
  int done;    // 1 once the iteration has converged and its last step is taken
  int extra;   // steps still to take after the switch (-1 before it)
  int iters;   // steps taken
  int pad;
  double res;  // last residual |I - P|_F
};

struct GemmArgs {
  int m, n;
  long long k;
  const double* A;
  long long lda;
  const double* B;
  long long ldb;
  const double* C;  // read when beta != 0 (may alias D)
  long long ldc;
  double* D;
  long long ldd;
  double alpha, beta, gamma;  // D = alpha * op(A) op(B) + beta * C + gamma * I
  const double* alpha_dev;    // multiplies alpha, or nullptr
  const int* skip;            // nothing is done while *skip != 0, or nullptr
};

// Stage one kBK x kBM slice of op(A) (As[kk][i]) and op(B) (Bs[kk][j]) in
// registers: each of the 256 threads holds 4 elements of each.
template <bool AK, bool BK>
__device__ inline void gemm_load(const GemmArgs& g, int m0, int n0, long long k0, int tid,
                                 double (&ra)[4], double (&rb)[4]) {
  if (AK) {  // op(A)(i, kk) = A[kk * lda + i]
    const int kk = tid >> 4, i4 = (tid & 15) * 4;
    const long long row = k0 + kk;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int i = m0 + i4 + e;
      ra[e] = (row < g.k && i < g.m) ? g.A[row * g.lda + i] : 0.0;
    }
  } else {  // op(A)(i, kk) = A[i * lda + kk]
    const int i = m0 + (tid >> 2), k4 = (tid & 3) * 4;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const long long kk = k0 + k4 + e;
      ra[e] = (i < g.m && kk < g.k) ? g.A[(long long)i * g.lda + kk] : 0.0;
    }
  }
  if (BK) {  // op(B)(kk, j) = B[kk * ldb + j]
    const int kk = tid >> 4, j4 = (tid & 15) * 4;
    const long long row = k0 + kk;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int j = n0 + j4 + e;
      rb[e] = (row < g.k && j < g.n) ? g.B[row * g.ldb + j] : 0.0;
    }
  } else {  // op(B)(kk, j) = B[j * ldb + kk]
    const int j = n0 + (tid >> 2), k4 = (tid & 3) * 4;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const long long kk = k0 + k4 + e;
      rb[e] = (j < g.n && kk < g.k) ? g.B[(long long)j * g.ldb + kk] : 0.0;
    }
  }
}

template <bool AK, bool BK>
__device__ inline void gemm_store(double (*As)[kBM + kPad], double (*Bs)[kBN + kPad], int tid,
                                  const double (&ra)[4], const double (&rb)[4]) {
  if (AK) {
    const int kk = tid >> 4, i4 = (tid & 15) * 4;
#pragma unroll
    for (int e = 0; e < 4; ++e) As[kk][i4 + e] = ra[e];
  } else {
    const int i = tid >> 2, k4 = (tid & 3) * 4;
#pragma unroll
    for (int e = 0; e < 4; ++e) As[k4 + e][i] = ra[e];
  }
  if (BK) {
    const int kk = tid >> 4, j4 = (tid & 15) * 4;
#pragma unroll
    for (int e = 0; e < 4; ++e) Bs[kk][j4 + e] = rb[e];
  } else {
    const int j = tid >> 2, k4 = (tid & 3) * 4;
#pragma unroll
    for (int e = 0; e < 4; ++e) Bs[k4 + e][j] = rb[e];
  }
}

// One 64 x 64 tile of D per workgroup; 4 waves in a 2 x 2 grid, each owning a
// 32 x 32 block as 2 x 2 matrix-core tiles of 16 x 16.  The fp64 MFMA reads
// op(A)(i, k) from lane i + 16 k and op(B)(k, j) from lane j + 16 k, and leaves
// D(lane / 16 + 4 v, lane % 16) in element v of each lane (rows interleaved).
template <bool AK, bool BK>
__global__ __launch_bounds__(kGemmThreads) void gemm_f64_kernel(GemmArgs g) {
  if (g.skip && *g.skip) return;
  const int tm = blockIdx.y, tn = blockIdx.x;
  __shared__ double As[2][kBK][kBM + kPad];
  __shared__ double Bs[2][kBK][kBN + kPad];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = tm * kBM, n0 = tn * kBN;
  const long long nk = (g.k + kBK - 1) / kBK;

  double4_t acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = double4_t{0.0, 0.0, 0.0, 0.0};

  double ra[4], rb[4];
  if (nk > 0) {
    gemm_load<AK, BK>(g, m0, n0, 0, tid, ra, rb);
    gemm_store<AK, BK>(As[0], Bs[0], tid, ra, rb);
  }
  __syncthreads();
  const int li = lane & 15, lk = lane >> 4;
  for (long long kt = 0; kt < nk; ++kt) {
    const int cur = (int)(kt & 1);
    const bool more = kt + 1 < nk;
    if (more) gemm_load<AK, BK>(g, m0, n0, (kt + 1) * kBK, tid, ra, rb);
#pragma unroll
    for (int ks = 0; ks < kBK / 4; ++ks) {
      double a[2], b[2];
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        a[x] = As[cur][ks * 4 + lk][wm * 32 + x * 16 + li];
        b[x] = Bs[cur][ks * 4 + lk][wn * 32 + x * 16 + li];
      }
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[x], b[y], acc[x][y], 0, 0, 0);
    }
    if (more) gemm_store<AK, BK>(As[cur ^ 1], Bs[cur ^ 1], tid, ra, rb);
    __syncthreads();
  }

  const double alpha = g.alpha_dev ? g.alpha * *g.alpha_dev : g.alpha;
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = m0 + wm * 32 + x * 16 + lk + 4 * v;
        const int j = n0 + wn * 32 + y * 16 + li;
        if (i >= g.m || j >= g.n) continue;
        double val = alpha * acc[x][y][v];
        if (g.beta != 0.0) val += g.beta * g.C[(long long)i * g.ldc + j];
        if (i == j) val += g.gamma;
        g.D[(long long)i * g.ldd + j] = val;
      }
}

// ---------------------------------------------------------------------------
// Weighted, centred Gram product of the samples V = [X | Y] (n rows, m = p + q
// columns): G = (V - 1 shift^T)^T diag(w) (V - 1 shift^T), upper 128 x 128
// tiles only, the rows split into `splits` ranges whose partial tiles a second
// kernel adds up in a fixed order.  Work item = (split, tile), split-major, so
// the workgroups resident together stream the same rows.
// ---------------------------------------------------------------------------
constexpr int kCT = 128;   // tile edge
constexpr int kCK = 16;    // rows per step
constexpr int kCPad = 4;
constexpr int kCovResident = 512;  // workgroups resident at once (2 per CU)

struct CovArgs {
  long long n;
  int p, m;
  const void* X;
  long long ldx;
  const void* Y;
  long long ldy;
  const float* w;
  const double* shift;  // [m]
  int nt;               // tiles per edge
  int n_tiles;          // nt (nt + 1) / 2
  long long rows_per_split;
  int vec;              // column groups of 8 are 16-byte aligned and never straddle X | Y
  double* partial;      // [splits][n_tiles][kCT][kCT]
};

__device__ inline void load8(const float* p, float (&v)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ inline void load8(const uint16_t* p, float (&v)[8]) {
  const uint4 a = *reinterpret_cast<const uint4*>(p);
  const uint32_t u[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[2 * e] = __uint_as_float(u[e] << 16);
    v[2 * e + 1] = __uint_as_float(u[e] & 0xffff0000u);
  }
}
__device__ inline float load1(const float* p) { return *p; }
__device__ inline double load_elem(const float* p, long long i) { return (double)p[i]; }
__device__ inline double load_elem(const uint16_t* p, long long i) {
  return (double)__uint_as_float(((uint32_t)p[i]) << 16);
}
__device__ inline float load1(const uint16_t* p) { return __uint_as_float(((uint32_t)*p) << 16); }

// Eight consecutive columns c0..c0+7 of sample row r (zeros past m).
template <typename T>
__device__ inline void cov_load(const CovArgs& g, long long r, int c0, float (&v)[8]) {
  const T* X = static_cast<const T*>(g.X);
  const T* Y = static_cast<const T*>(g.Y);
  if (g.vec) {
    if (c0 >= g.m) {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = 0.f;
    } else if (c0 < g.p) {
      load8(X + r * g.ldx + c0, v);
    } else {
      load8(Y + r * g.ldy + (c0 - g.p), v);
    }
    return;
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int c = c0 + e;
    v[e] = c >= g.m ? 0.f : (c < g.p ? load1(X + r * g.ldx + c) : load1(Y + r * g.ldy + (c - g.p)));
  }
}

// 256 threads = 4 waves in a 2 x 2 grid, each owning 64 x 64 as 4 x 4 MFMA tiles.
template <typename T>
__global__ __launch_bounds__(256) void cov_kernel(CovArgs g) {
  __shared__ double As[2][kCK][kCT + kCPad];
  __shared__ double Bs[2][kCK][kCT + kCPad];
  const int item = blockIdx.x;
  const int split = item / g.n_tiles, tile = item - split * g.n_tiles;
  int tm = 0, rem = tile;
  while (rem >= g.nt - tm) {
    rem -= g.nt - tm;
    ++tm;
  }
  const int tn = tm + rem;
  const long long r_beg = (long long)split * g.rows_per_split;
  const long long r_end = r_beg + g.rows_per_split < g.n ? r_beg + g.rows_per_split : g.n;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int li = lane & 15, lk = lane >> 4;

  // staging role: one row (kk) and eight consecutive columns (c8) of each operand
  const int kk = tid >> 4, c8 = (tid & 15) * 8;
  const int ca = tm * kCT + c8, cb = tn * kCT + c8;
  double sha[8], shb[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    sha[e] = ca + e < g.m ? g.shift[ca + e] : 0.0;
    shb[e] = cb + e < g.m ? g.shift[cb + e] : 0.0;
  }

  double4_t acc[4][4];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) acc[x][y] = double4_t{0.0, 0.0, 0.0, 0.0};

  float va[8], vb[8];
  float wr = 0.f;
  auto fetch = [&](long long k0) {
    const long long r = k0 + kk;
    if (r < r_end) {
      cov_load<T>(g, r, ca, va);
      cov_load<T>(g, r, cb, vb);
      wr = g.w ? g.w[r] : 1.f;
    } else {
      wr = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) va[e] = vb[e] = 0.f;
    }
  };
  auto stage = [&](int buf) {
    const double wd = (double)wr;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      // rows past the range carry weight 0 on the A side and stage 0 on the B side
      As[buf][kk][c8 + e] = ((double)va[e] - sha[e]) * wd;
      Bs[buf][kk][c8 + e] = wr != 0.f ? (double)vb[e] - shb[e] : 0.0;
    }
  };

  const long long nk = (r_end - r_beg + kCK - 1) / kCK;
  if (nk > 0) {
    fetch(r_beg);
    stage(0);
  }
  __syncthreads();
  for (long long kt = 0; kt < nk; ++kt) {
    const int cur = (int)(kt & 1);
    const bool more = kt + 1 < nk;
    if (more) fetch(r_beg + (kt + 1) * kCK);
#pragma unroll
    for (int ks = 0; ks < kCK / 4; ++ks) {
      double a[4], b[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        a[x] = As[cur][ks * 4 + lk][wm * 64 + x * 16 + li];
        b[x] = Bs[cur][ks * 4 + lk][wn * 64 + x * 16 + li];
      }
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[x], b[y], acc[x][y], 0, 0, 0);
    }
    if (more) stage(cur ^ 1);
    __syncthreads();
  }

  double* out = g.partial + ((long long)split * g.n_tiles + tile) * (kCT * kCT);
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        out[(wm * 64 + x * 16 + lk + 4 * v) * kCT + wn * 64 + y * 16 + li] = acc[x][y][v];
}

// cov[i][j] = scale_i scale_j / W * sum over splits of the (min, max) entry:
// both triangles from the upper tiles, so the result is exactly symmetric.
__global__ __launch_bounds__(256) void cov_reduce_kernel(const double* partial, int splits,
                                                          int n_tiles, int nt, int m,
                                                          const double* scale,
                                                          const double* inv_w, double* cov) {
  const long long total = (long long)m * m;
  const double iw = *inv_w;
  for (long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (long long)gridDim.x * blockDim.x) {
    const int i = (int)(e / m), j = (int)(e - (long long)i * m);
    const int a = i < j ? i : j, b = i < j ? j : i;
    const int tm = a / kCT, tn = b / kCT;
    const long long tile = (long long)tm * nt - (long long)tm * (tm - 1) / 2 + (tn - tm);
    const long long off = tile * (kCT * kCT) + (a - tm * kCT) * kCT + (b - tn * kCT);
    double s = 0.0;
    for (int k = 0; k < splits; ++k) s += partial[(long long)k * n_tiles * (kCT * kCT) + off];
    cov[e] = s * scale[i] * scale[j] * iw;
  }
}

// ---------------------------------------------------------------------------
// Reductions (fixed order: block tree, then one block over the partials).
// ---------------------------------------------------------------------------
__device__ inline double block_sum(double v, double* red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  double s = 0.0;
  if (threadIdx.x == 0)
    for (int i = 0; i < (int)(blockDim.x >> 6); ++i) s += red[i];
  return s;  // valid in thread 0
}

// partial[block] = sum over its share of (M[i][j] + add * [i == j])^2
__global__ __launch_bounds__(kRedThreads) void sumsq_kernel(const double* M, int rows, int cols,
                                                             long long ld, const double* add_dev,
                                                             const int* skip, double* partial) {
  if (skip && *skip) return;
  __shared__ double red[kRedThreads / 64];
  const double add = add_dev ? *add_dev : 0.0;
  const long long total = (long long)rows * cols;
  double s = 0.0;
  for (long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (long long)gridDim.x * blockDim.x) {
    const int i = (int)(e / cols), j = (int)(e - (long long)i * cols);
    const double v = M[(long long)i * ld + j] + (i == j ? add : 0.0);
    s += v * v;
  }
  s = block_sum(s, red);
  if (threadIdx.x == 0) partial[blockIdx.x] = s;
}

__device__ inline double sum_partials(const double* partial, int n, double* red) {
  double s = 0.0;
  for (int i = threadIdx.x; i < n; i += blockDim.x) s += partial[i];
  return block_sum(s, red);
}

// out = sqrt(sum of partials)
__global__ __launch_bounds__(kRedThreads) void frob_finish_kernel(const double* partial, int n,
                                                                   const int* skip, double* out) {
  if (skip && *skip) return;
  __shared__ double red[kRedThreads / 64];
  const double s = sum_partials(partial, n, red);
  if (threadIdx.x == 0) *out = sqrt(s);
}

// Newton-Schulz step decision from the residual |I - P|_F = 2 |T - I|_F.
__global__ __launch_bounds__(kRedThreads) void ns_check_kernel(const double* partial, int n,
                                                                NsState* st) {
  if (st->done) return;
  __shared__ double red[kRedThreads / 64];
  const double s = sum_partials(partial, n, red);
  if (threadIdx.x != 0) return;
  const double res = 2.0 * sqrt(s);
  st->res = res;
  if (st->extra == 0) {
    st->done = 1;
    return;
  }
  if (st->extra > 0)
    st->extra -= 1;
  else if (res <= kNsSwitch)
    st->extra = kNsExtra;
  st->iters += 1;
}

// ridge: *lam_abs = lam * trace(M) / d over M's leading d x d block
__global__ __launch_bounds__(kRedThreads) void ridge_kernel(const double* M, long long ld, int d,
                                                             double lam, double* lam_abs) {
  __shared__ double red[kRedThreads / 64];
  double s = 0.0;
  for (int i = threadIdx.x; i < d; i += blockDim.x) s += M[(long long)i * ld + i];
  s = block_sum(s, red);
  if (threadIdx.x == 0) *lam_abs = lam * s / d;
}

// Y = (M + lam_abs I) / c, Z = I
__global__ void ns_sqrt_init_kernel(const double* M, long long ld, int d, const double* lam_abs,
                                    const double* c, double* Y, double* Z) {
  const long long total = (long long)d * d;
  const double inv = 1.0 / *c, lam = *lam_abs;
  for (long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (long long)gridDim.x * blockDim.x) {
    const int i = (int)(e / d), j = (int)(e - (long long)i * d);
    Y[e] = (M[(long long)i * ld + j] + (i == j ? lam : 0.0)) * inv;
    Z[e] = i == j ? 1.0 : 0.0;
  }
}

// X *= 1 / *nrm
__global__ void scale_kernel(double* X, long long total, const double* nrm) {
  const double inv = 1.0 / *nrm;
  for (long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (long long)gridDim.x * blockDim.x)
    X[e] *= inv;
}

// An odd number of ping-pong steps leaves the iterate in buffer 1: move it to 0.
__global__ void ns_settle_kernel(const NsState* st, const double* src, double* dst,
                                 long long total) {
  if ((st->iters & 1) == 0) return;
  for (long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (long long)gridDim.x * blockDim.x)
    dst[e] = src[e];
}

__global__ void ns_reset_kernel(NsState* st, int n) {
  const int i = threadIdx.x;
  if (i < n) {
    st[i].done = 0;
    st[i].extra = -1;
    st[i].iters = 0;
    st[i].pad = 0;
    st[i].res = -1.0;
  }
}

__global__ void ratio_sqrt_kernel(const double* num, const double* den, double* out) {
  if (threadIdx.x == 0) *out = sqrt(*num / *den);
}

__global__ void info_kernel(const NsState* st, hf_recolor_info* info) {
  const int i = threadIdx.x;
  if (i < 3) {
    info->iterations[i] = st[i].iters;
    info->converged[i] = st[i].done;
    info->residual[i] = st[i].res;
  }
}

// ---------------------------------------------------------------------------
// Column statistics of the samples: weighted sums per column and the weighted
// sum of squares of the X columns, per chunk of rows.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void colstats_kernel(long long n, int p, int q, const T* X,
                                                        long long ldx, const T* Y, long long ldy,
                                                        const float* w, long long rows_per_chunk,
                                                        double* part_sum, double* part_sq,
                                                        double* part_w) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  const int chunk = blockIdx.y;
  const long long r0 = (long long)chunk * rows_per_chunk;
  const long long r1 = r0 + rows_per_chunk < n ? r0 + rows_per_chunk : n;
  const int pq = p + q;
  if (c < pq) {
    double s = 0.0, ss = 0.0;
    for (long long r = r0; r < r1; ++r) {
      const double wv = w ? (double)w[r] : 1.0;
      const double v = c < p ? load_elem(X, r * ldx + c) : load_elem(Y, r * ldy + (c - p));
      s += wv * v;
      ss += wv * v * v;
    }
    part_sum[(long long)chunk * pq + c] = s;
    if (c < p) part_sq[(long long)chunk * p + c] = ss;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    double sw = 0.0;
    for (long long r = r0; r < r1; ++r) sw += w ? (double)w[r] : 1.0;
    part_w[chunk] = sw;
  }
}

// Per column: total weighted sum and (X columns) sum of squares over the chunks.
__global__ __launch_bounds__(256) void colstats_reduce_kernel(int p, int q, int n_chunks,
                                                               const double* part_sum,
                                                               const double* part_sq,
                                                               double* col_sum, double* col_sq) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  const int pq = p + q;
  if (c >= pq) return;
  double s = 0.0, ss = 0.0;
  for (int k = 0; k < n_chunks; ++k) {
    s += part_sum[(long long)k * pq + c];
    if (c < p) ss += part_sq[(long long)k * p + c];
  }
  col_sum[c] = s;
  if (c < p) col_sq[c] = ss;
}

// W, r (Eq. 3), raw means (centring shifts), column scales (1/r for X, 1 for
// Y), the means of [x/r | y], and 1/W.
__global__ __launch_bounds__(kRedThreads) void moments_scalars_kernel(
    int p, int q, int n_chunks, const double* part_w, const double* col_sum, const double* col_sq,
    double* shift, double* scale, double* mu, double* r_out, double* inv_w) {
  __shared__ double red[kRedThreads / 64];
  __shared__ double sh_w, sh_r;
  const double W = sum_partials(part_w, n_chunks, red);
  double s = 0.0;
  for (int c = threadIdx.x; c < p; c += blockDim.x) s += col_sq[c];
  s = block_sum(s, red);
  if (threadIdx.x == 0) {
    sh_w = W;
    sh_r = sqrt(s / ((double)p * W));
    *r_out = sh_r;
    *inv_w = 1.0 / W;
  }
  __syncthreads();
  const double Wv = sh_w, rv = sh_r;
  for (int c = threadIdx.x; c < p + q; c += blockDim.x) {
    const double m = col_sum[c] / Wv;
    shift[c] = m;
    scale[c] = c < p ? 1.0 / rv : 1.0;
    mu[c] = c < p ? m / rv : m;
  }
}

int grid_for(long long total, int threads = 256, int cap = 4096) {
  long long b = (total + threads - 1) / threads;
  if (b < 1) b = 1;
  return (int)(b < cap ? b : cap);
}

template <bool AK, bool BK>
hipError_t gemm_launch(const GemmArgs& g, hipStream_t s) {
  dim3 grid((g.n + kBN - 1) / kBN, (g.m + kBM - 1) / kBM);
  hipLaunchKernelGGL((gemm_f64_kernel<AK, BK>), grid, dim3(kGemmThreads), 0, s, g);
  return hipGetLastError();
}

// Plain fp64 product D = alpha * op(A) op(B) + beta * C + gamma * I with
// op(A) m x k (ak: stored k-major, A[kk * lda + i]) and op(B) k x n (bk: stored
// k-major, B[kk * ldb + j]).
hipError_t gemm(int m, int n, long long k, const double* A, long long lda, bool ak,
                const double* B, long long ldb, bool bk, double* D, long long ldd,
                hipStream_t s, double alpha = 1.0, double beta = 0.0, const double* C = nullptr,
                long long ldc = 0, double gamma = 0.0, const double* alpha_dev = nullptr,
                const int* skip = nullptr) {
  GemmArgs g{};
  g.m = m;
  g.n = n;
  g.k = k;
  g.A = A;
  g.lda = lda;
  g.B = B;
  g.ldb = ldb;
  g.C = C;
  g.ldc = ldc;
  g.D = D;
  g.ldd = ldd;
  g.alpha = alpha;
  g.beta = beta;
  g.gamma = gamma;
  g.alpha_dev = alpha_dev;
  g.skip = skip;
  if (ak && bk) return gemm_launch<true, true>(g, s);
  if (ak) return gemm_launch<true, false>(g, s);
  if (bk) return gemm_launch<false, true>(g, s);
  return gemm_launch<false, false>(g, s);
}

#define HF_CHECK(x)                   \
  do {                                \
    hipError_t e_ = (x);              \
    if (e_ != hipSuccess) return e_;  \
  } while (0)

// Scratch carving from the workspace (256-byte aligned pieces).
struct Carve {
  char* p;
  template <typename U>
  U* take(size_t count) {
    U* r = reinterpret_cast<U*>(p);
    p += (count * sizeof(U) + 255) / 256 * 256;
    return r;
  }
};

constexpr int kSqrtMaxIter = 64;    // even: the ping-pong pairs stay aligned
constexpr int kPolarMaxIter = 128;

// Coupled Newton-Schulz iteration on S = M + lam_abs I (d x d, SPD):
//   Y0 = S / c, Z0 = I, T = (3I - Z Y) / 2, Y <- Y T, Z <- T Z,
// Y -> (S/c)^{1/2}, Z -> (S/c)^{-1/2}, with c = |S|_F.  Results in Y[0], Z[0].
hipError_t ns_sqrt(const double* M, long long ld, int d, double lam, double* Y[2], double* Z[2],
                   double* T, double* partial, double* lam_abs, double* c,
                   const double* minus_one, NsState* st, hipStream_t s) {
  hipLaunchKernelGGL(ridge_kernel, dim3(1), dim3(kRedThreads), 0, s, M, ld, d, lam, lam_abs);
  HF_CHECK(hipGetLastError());
  const long long dd = (long long)d * d;
  const int nred = grid_for(dd, kRedThreads, kMaxRedBlocks);
  hipLaunchKernelGGL(sumsq_kernel, dim3(nred), dim3(kRedThreads), 0, s, M, d, d, ld,
                     (const double*)lam_abs, (const int*)nullptr, partial);
  HF_CHECK(hipGetLastError());
  hipLaunchKernelGGL(frob_finish_kernel, dim3(1), dim3(kRedThreads), 0, s, (const double*)partial,
                     nred, (const int*)nullptr, c);
  HF_CHECK(hipGetLastError());
  hipLaunchKernelGGL(ns_sqrt_init_kernel, dim3(grid_for(dd)), dim3(256), 0, s, M, ld, d,
                     (const double*)lam_abs, (const double*)c, Y[0], Z[0]);
  HF_CHECK(hipGetLastError());
  const int* skip = &st->done;
  for (int it = 0; it < kSqrtMaxIter; ++it) {
    const int a = it & 1, b = a ^ 1;
    // T = -1/2 Z Y + 3/2 I
    HF_CHECK(gemm(d, d, d, Z[a], d, false, Y[a], d, true, T, d, s, -0.5, 0.0, nullptr, 0, 1.5,
                  nullptr, skip));
    hipLaunchKernelGGL(sumsq_kernel, dim3(nred), dim3(kRedThreads), 0, s, (const double*)T, d, d,
                       (long long)d, minus_one, skip, partial);
    HF_CHECK(hipGetLastError());
    hipLaunchKernelGGL(ns_check_kernel, dim3(1), dim3(kRedThreads), 0, s, (const double*)partial,
                       nred, st);
    HF_CHECK(hipGetLastError());
    HF_CHECK(gemm(d, d, d, Y[a], d, false, T, d, true, Y[b], d, s, 1.0, 0.0, nullptr, 0, 0.0,
                  nullptr, skip));
    HF_CHECK(gemm(d, d, d, T, d, false, Z[a], d, true, Z[b], d, s, 1.0, 0.0, nullptr, 0, 0.0,
                  nullptr, skip));
  }
  hipLaunchKernelGGL(ns_settle_kernel, dim3(grid_for(dd)), dim3(256), 0, s, (const NsState*)st,
                     (const double*)Y[1], Y[0], dd);
  HF_CHECK(hipGetLastError());
  hipLaunchKernelGGL(ns_settle_kernel, dim3(grid_for(dd)), dim3(256), 0, s, (const NsState*)st,
                     (const double*)Z[1], Z[0], dd);
  return hipGetLastError();
}

// Newton-Schulz iteration for the polar factor of the p x q matrix in X[0]:
// X0 = M / |M|_F, then X <- X (3I - X^T X) / 2 (p >= q) or X <- (3I - X X^T) X / 2
// (p < q).  Result in X[0].
hipError_t ns_polar(int p, int q, double* X[2], double* T, double* partial, double* nrm,
                    const double* minus_one, NsState* st, hipStream_t s) {
  const long long pq = (long long)p * q;
  const int nred_m = grid_for(pq, kRedThreads, kMaxRedBlocks);
  hipLaunchKernelGGL(sumsq_kernel, dim3(nred_m), dim3(kRedThreads), 0, s, (const double*)X[0], p,
                     q, (long long)q, (const double*)nullptr, (const int*)nullptr, partial);
  HF_CHECK(hipGetLastError());
  hipLaunchKernelGGL(frob_finish_kernel, dim3(1), dim3(kRedThreads), 0, s, (const double*)partial,
                     nred_m, (const int*)nullptr, nrm);
  HF_CHECK(hipGetLastError());
  hipLaunchKernelGGL(scale_kernel, dim3(grid_for(pq)), dim3(256), 0, s, X[0], pq,
                     (const double*)nrm);
  HF_CHECK(hipGetLastError());
  const int e = p >= q ? q : p;
  const long long ee = (long long)e * e;
  const int nred = grid_for(ee, kRedThreads, kMaxRedBlocks);
  const int* skip = &st->done;
  for (int it = 0; it < kPolarMaxIter; ++it) {
    const int a = it & 1, b = a ^ 1;
    if (p >= q) {
      // T = -1/2 X^T X + 3/2 I (q x q); X' = X T
      HF_CHECK(gemm(q, q, p, X[a], q, true, X[a], q, true, T, q, s, -0.5, 0.0, nullptr, 0, 1.5,
                    nullptr, skip));
    } else {
      // T = -1/2 X X^T + 3/2 I (p x p); X' = T X
      HF_CHECK(gemm(p, p, q, X[a], q, false, X[a], q, false, T, p, s, -0.5, 0.0, nullptr, 0, 1.5,
                    nullptr, skip));
    }
    hipLaunchKernelGGL(sumsq_kernel, dim3(nred), dim3(kRedThreads), 0, s, (const double*)T, e, e,
                       (long long)e, minus_one, skip, partial);
    HF_CHECK(hipGetLastError());
    hipLaunchKernelGGL(ns_check_kernel, dim3(1), dim3(kRedThreads), 0, s, (const double*)partial,
                       nred, st);
    HF_CHECK(hipGetLastError());
    if (p >= q)
      HF_CHECK(gemm(p, q, q, X[a], q, false, T, q, true, X[b], q, s, 1.0, 0.0, nullptr, 0, 0.0,
                    nullptr, skip));
    else
      HF_CHECK(gemm(p, q, p, T, p, false, X[a], q, true, X[b], q, s, 1.0, 0.0, nullptr, 0, 0.0,
                    nullptr, skip));
  }
  hipLaunchKernelGGL(ns_settle_kernel, dim3(grid_for(pq)), dim3(256), 0, s, (const NsState*)st,
                     (const double*)X[1], X[0], pq);
  return hipGetLastError();
}

// Scalar slots of the solve's workspace.
enum {
  kScLamZ = 0,
  kScLamY = 1,
  kScCZ = 2,
  kScCY = 3,
  kScNormM = 4,
  kScAlphaA = 5,
  kScMinusOne = 6,  // the residual kernels subtract I through their "add" value
  kScCount = 16
};

__global__ void solve_consts_kernel(double* sc) {
  if (threadIdx.x == 0) sc[kScMinusOne] = -1.0;
}

}  // namespace

int moments_chunks(long long n) {
  long long c = (n + 255) / 256;
  if (c > 512) c = 512;
  if (c < 1) c = 1;
  return (int)c;
}

namespace {

struct CovPlan {
  int nt, n_tiles, splits;
  long long rows_per_split;
};

// Rows are split so that the (split, tile) items fill the resident workgroups
// with the least idle tail, each split keeping at least 32 steps of rows.
CovPlan cov_plan(long long n, int m) {
  CovPlan c;
  c.nt = (m + kCT - 1) / kCT;
  c.n_tiles = c.nt * (c.nt + 1) / 2;
  const long long steps = (n + kCK - 1) / kCK;
  long long max_splits = steps / 32;
  if (max_splits < 1) max_splits = 1;
  if (max_splits > 64) max_splits = 64;
  int best = 1;
  double best_waste = 1e30;
  for (int s = 1; s <= max_splits; ++s) {
    const long long items = (long long)s * c.n_tiles;
    if (items < kCovResident && s < max_splits) continue;
    const long long rounds = (items + kCovResident - 1) / kCovResident;
    const double waste = (double)(rounds * kCovResident) / (double)items - 1.0;
    if (waste < best_waste - 0.01) {
      best_waste = waste;
      best = s;
    }
  }
  c.splits = best;
  c.rows_per_split = (steps + best - 1) / best * kCK;
  return c;
}

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

}  // namespace

size_t recolor_moments_workspace_bytes(long long n, int p, int q) {
  const size_t n_chunks = (size_t)moments_chunks(n);
  const size_t pq = (size_t)p + q;
  const CovPlan c = cov_plan(n, p + q);
  return align256(n_chunks * pq * 8) + align256(n_chunks * (size_t)p * 8) +
         align256(n_chunks * 8) + align256(pq * 8) + align256((size_t)p * 8) +
         2 * align256(pq * 8) + align256(8) +
         align256((size_t)c.splits * c.n_tiles * kCT * kCT * 8);
}

hipError_t launch_recolor_stats(int dtype, long long n, int p, int q, const void* X,
                                long long ldx, const void* Y, long long ldy, const float* w,
                                double* r, double* mu, void* workspace, hipStream_t s) {
  const int n_chunks = moments_chunks(n);
  const long long rows_per_chunk = (n + n_chunks - 1) / n_chunks;
  const int pq = p + q;
  Carve cv{static_cast<char*>(workspace)};
  double* part_sum = cv.take<double>((size_t)n_chunks * pq);
  double* part_sq = cv.take<double>((size_t)n_chunks * p);
  double* part_w = cv.take<double>(n_chunks);
  double* col_sum = cv.take<double>(pq);
  double* col_sq = cv.take<double>(p);
  double* shift = cv.take<double>(pq);
  double* scale = cv.take<double>(pq);
  double* inv_w = cv.take<double>(1);

  dim3 g1((pq + 255) / 256, n_chunks);
  if (dtype == HF_BF16)
    hipLaunchKernelGGL(colstats_kernel<uint16_t>, g1, dim3(256), 0, s, n, p, q,
                       static_cast<const uint16_t*>(X), ldx, static_cast<const uint16_t*>(Y), ldy,
                       w, rows_per_chunk, part_sum, part_sq, part_w);
  else
    hipLaunchKernelGGL(colstats_kernel<float>, g1, dim3(256), 0, s, n, p, q,
                       static_cast<const float*>(X), ldx, static_cast<const float*>(Y), ldy, w,
                       rows_per_chunk, part_sum, part_sq, part_w);
  HF_CHECK(hipGetLastError());
  hipLaunchKernelGGL(colstats_reduce_kernel, dim3((pq + 255) / 256), dim3(256), 0, s, p, q,
                     n_chunks, (const double*)part_sum, (const double*)part_sq, col_sum, col_sq);
  HF_CHECK(hipGetLastError());
  hipLaunchKernelGGL(moments_scalars_kernel, dim3(1), dim3(kRedThreads), 0, s, p, q, n_chunks,
                     (const double*)part_w, (const double*)col_sum, (const double*)col_sq, shift,
                     scale, mu, r, inv_w);
  HF_CHECK(hipGetLastError());
  return hipSuccess;
}

hipError_t launch_recolor_cov(int dtype, long long n, int p, int q, const void* X, long long ldx,
                              const void* Y, long long ldy, const float* w, void* workspace,
                              hipStream_t s) {
  const int n_chunks = moments_chunks(n);
  const int pq = p + q;
  Carve cv{static_cast<char*>(workspace)};
  (void)cv.take<double>((size_t)n_chunks * pq);
  (void)cv.take<double>((size_t)n_chunks * p);
  (void)cv.take<double>(n_chunks);
  (void)cv.take<double>(pq);
  (void)cv.take<double>(p);
  double* shift = cv.take<double>(pq);
  (void)cv.take<double>(pq);  // column scales (applied by the reduction)
  (void)cv.take<double>(1);   // 1 / W
  const CovPlan plan = cov_plan(n, pq);
  double* partial = cv.take<double>((size_t)plan.splits * plan.n_tiles * kCT * kCT);
  CovArgs g{};
  g.n = n;
  g.p = p;
  g.m = pq;
  g.X = X;
  g.ldx = ldx;
  g.Y = Y;
  g.ldy = ldy;
  g.w = w;
  g.shift = shift;
  g.nt = plan.nt;
  g.n_tiles = plan.n_tiles;
  g.rows_per_split = plan.rows_per_split;
  g.partial = partial;
  const int per16 = dtype == HF_BF16 ? 8 : 4;  // elements per 16 bytes
  g.vec = (p % 8 == 0) && (q % 8 == 0) && (ldx % per16 == 0) && (ldy % per16 == 0) &&
          ((uintptr_t)X % 16 == 0) && ((uintptr_t)Y % 16 == 0);
  const unsigned items = (unsigned)((long long)plan.splits * plan.n_tiles);
  if (dtype == HF_BF16)
    hipLaunchKernelGGL(cov_kernel<uint16_t>, dim3(items), dim3(256), 0, s, g);
  else
    hipLaunchKernelGGL(cov_kernel<float>, dim3(items), dim3(256), 0, s, g);
  return hipGetLastError();
}

hipError_t launch_recolor_cov_reduce(long long n, int p, int q, double* cov, void* workspace,
                                     hipStream_t s) {
  const int n_chunks = moments_chunks(n);
  const int pq = p + q;
  Carve cv{static_cast<char*>(workspace)};
  (void)cv.take<double>((size_t)n_chunks * pq);
  (void)cv.take<double>((size_t)n_chunks * p);
  (void)cv.take<double>(n_chunks);
  (void)cv.take<double>(pq);
  (void)cv.take<double>(p);
  (void)cv.take<double>(pq);
  double* scale = cv.take<double>(pq);
  double* inv_w = cv.take<double>(1);
  const CovPlan plan = cov_plan(n, pq);
  double* partial = cv.take<double>((size_t)plan.splits * plan.n_tiles * kCT * kCT);
  hipLaunchKernelGGL(cov_reduce_kernel, dim3(grid_for((long long)pq * pq, 256, 8192)), dim3(256),
                     0, s, (const double*)partial, plan.splits, plan.n_tiles, plan.nt, pq,
                     (const double*)scale, (const double*)inv_w, cov);
  return hipGetLastError();
}

size_t recolor_solve_workspace_bytes(int p, int q) {
  auto a = [](size_t b) { return (b + 255) / 256 * 256; };
  const size_t pp = (size_t)p * p, qq = (size_t)q * q, pq = (size_t)p * q;
  const size_t e = p < q ? p : q;
  return a(kScCount * 8) + a(3 * sizeof(NsState)) + a(kMaxRedBlocks * 8) + 5 * a(pp * 8) +
         5 * a(qq * 8) + 2 * a(pq * 8) + a(e * e * 8) + a(pq * 8) + a(pq * 8);
}

hipError_t launch_recolor_solve(int p, int q, const double* mu, const double* cov, double lam,
                                double* A, double* b, hf_recolor_info* info, void* workspace,
                                hipStream_t s) {
  const int pq = p + q;
  Carve cv{static_cast<char*>(workspace)};
  double* sc = cv.take<double>(kScCount);
  NsState* st = cv.take<NsState>(3);
  double* partial = cv.take<double>(kMaxRedBlocks);
  double* Yz[2] = {cv.take<double>((size_t)p * p), cv.take<double>((size_t)p * p)};
  double* Zz[2] = {cv.take<double>((size_t)p * p), cv.take<double>((size_t)p * p)};
  double* Tz = cv.take<double>((size_t)p * p);
  double* Yy[2] = {cv.take<double>((size_t)q * q), cv.take<double>((size_t)q * q)};
  double* Zy[2] = {cv.take<double>((size_t)q * q), cv.take<double>((size_t)q * q)};
  double* Ty = cv.take<double>((size_t)q * q);
  double* Xp[2] = {cv.take<double>((size_t)p * q), cv.take<double>((size_t)p * q)};
  const size_t e = p < q ? p : q;
  double* Tp = cv.take<double>(e * e);
  double* Tmp1 = cv.take<double>((size_t)p * q);  // Z_z C (p x q)
  double* Tmp2 = cv.take<double>((size_t)p * q);  // R^T Z_z (q x p)

  hipLaunchKernelGGL(ns_reset_kernel, dim3(1), dim3(64), 0, s, st, 3);
  HF_CHECK(hipGetLastError());
  hipLaunchKernelGGL(solve_consts_kernel, dim3(1), dim3(64), 0, s, sc);
  HF_CHECK(hipGetLastError());
  HF_CHECK(ns_sqrt(cov, pq, p, lam, Yz, Zz, Tz, partial, sc + kScLamZ, sc + kScCZ,
                   sc + kScMinusOne, st + 0, s));
  HF_CHECK(ns_sqrt(cov + (long long)p * pq + p, pq, q, lam, Yy, Zy, Ty, partial, sc + kScLamY,
                   sc + kScCY, sc + kScMinusOne, st + 1, s));
  // M ~ Sigma_Z^{-1/2} Sigma_ZY Sigma_Y^{-1/2} (positive scale: the polar factor ignores it)
  HF_CHECK(gemm(p, q, p, Zz[0], p, false, cov + p, pq, true, Tmp1, q, s));
  HF_CHECK(gemm(p, q, q, Tmp1, q, false, Zy[0], q, true, Xp[0], q, s));
  HF_CHECK(ns_polar(p, q, Xp, Tp, partial, sc + kScNormM, sc + kScMinusOne, st + 2, s));
  // A (stored q x p) = Sigma_Y^{1/2} R^T Sigma_Z^{-1/2} = sqrt(c_Y / c_Z) Y_y R^T Z_z
  hipLaunchKernelGGL(ratio_sqrt_kernel, dim3(1), dim3(64), 0, s, (const double*)(sc + kScCY),
                     (const double*)(sc + kScCZ), sc + kScAlphaA);
  HF_CHECK(hipGetLastError());
  HF_CHECK(gemm(q, p, p, Xp[0], q, true, Zz[0], p, true, Tmp2, p, s));
  HF_CHECK(gemm(q, p, q, Yy[0], q, false, Tmp2, p, true, A, p, s, 1.0, 0.0, nullptr, 0, 0.0,
                sc + kScAlphaA));
  // b = mu_Y - A mu_Z
  HF_CHECK(gemm(q, 1, p, A, p, false, mu, 1, true, b, 1, s, -1.0, 1.0, mu + p, 1));
  if (info) {
    hipLaunchKernelGGL(info_kernel, dim3(1), dim3(64), 0, s, (const NsState*)st, info);
    HF_CHECK(hipGetLastError());
  }
  return hipSuccess;
}

size_t fold_workspace_bytes(int p, int rank) {
  return ((size_t)rank * p * 8 + 255) / 256 * 256 + ((size_t)rank * 8 + 255) / 256 * 256;
}

hipError_t launch_fold(int p, int q, int rank, const double* A, const double* b, const double* B,
                       const double* G, double* A_out, double* b_out, void* workspace,
                       hipStream_t s) {
  Carve cv{static_cast<char*>(workspace)};
  double* T = cv.take<double>((size_t)rank * p);
  double* t = cv.take<double>(rank);
  // stored maps: A_out = (I + B G)^T A = A + G^T (B^T A); same for the bias column
  HF_CHECK(gemm(rank, p, q, B, rank, true, A, p, true, T, p, s));
  HF_CHECK(gemm(rank, 1, q, B, rank, true, b, 1, true, t, 1, s));
  HF_CHECK(gemm(q, p, rank, G, q, true, T, p, true, A_out, p, s, 1.0, 1.0, A, p));
  HF_CHECK(gemm(q, 1, rank, G, q, true, t, 1, true, b_out, 1, s, 1.0, 1.0, b, 1));
  return hipSuccess;
}

hipError_t launch_gemm_f64(int m, int n, long long k, const double* A, long long lda, int ak,
                           const double* B, long long ldb, int bk, double* D, long long ldd,
                           double alpha, double beta, const double* C, long long ldc,
                           double gamma, hipStream_t s) {
  return gemm(m, n, k, A, lda, ak != 0, B, ldb, bk != 0, D, ldd, s, alpha, beta, C, ldc, gamma);
}

}  // namespace hf
