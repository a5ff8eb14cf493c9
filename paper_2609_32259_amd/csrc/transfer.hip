// KV transfer kernels: RoPE cos/sin tables, map packing, and the transfer
// itself (layer interpolation + RoPE un-rotation + overlap-weighted segment
// mean, then the folded affine map of Eq. 9 with bias and receiver RoPE in
// the epilogue, written straight into the receiver cache layout).
#include <hip/hip_runtime.h>

#include "hf_internal.h"

namespace hf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// ---------------------------------------------------------------------------
// bf16 helpers.  bf16 -> f32 is exact (the bf16 bits are the top half of the
// f32); f32 -> bf16 rounds to nearest even (v_cvt_pk_bf16_f32).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

__device__ __forceinline__ void unpack8(const uint4 v, float* f) {
  f[0] = bf_lo(v.x); f[1] = bf_hi(v.x);
  f[2] = bf_lo(v.y); f[3] = bf_hi(v.y);
  f[4] = bf_lo(v.z); f[5] = bf_hi(v.z);
  f[6] = bf_lo(v.w); f[7] = bf_hi(v.w);
}

__device__ __forceinline__ uint32_t pack2(float a, float b) {
  bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint4 pack8(const float* f) {
  return make_uint4(pack2(f[0], f[1]), pack2(f[2], f[3]), pack2(f[4], f[5]), pack2(f[6], f[7]));
}

// ---------------------------------------------------------------------------
// RoPE tables: tab[pos][k] = (cos, sin)(pos * theta^(-2k/d)), angle in fp64.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void rope_table_kernel(float2* tab, int P, int half, int d,
                                                         double theta) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long long)P * half) return;
  const int pos = (int)(idx / half), k = (int)(idx % half);
  const double w = pow(theta, -2.0 * k / d);
  const double ang = (double)pos * w;
  double s, c;
  sincos(ang, &s, &c);
  tab[idx] = make_float2((float)c, (float)s);
}

// ---------------------------------------------------------------------------
// Map packing for the bf16 matrix-core kernel.  One 1 KB fragment holds the
// 32 x 16 block (rows n, columns k) one v_mfma_f32_32x32x16_bf16 consumes as
// its A operand: lane l holds row n = 32 nb + l%32, columns
// k = 16 ks + 8 (l/32) + 0..7.  Fragments are ordered [lc][ks][nb], so a wave
// reads one fragment with a single fully coalesced 16-byte-per-lane load.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void pack_bf16_kernel(const uint16_t* A, uint4* Wp, long long n_frag_lanes,
                                                        int d_r, int d_in) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= n_frag_lanes) return;
  const int NB = d_r / 32, KS = d_in / 16;
  const int lane = (int)(idx & 63);
  long long t = idx >> 6;
  const int nb = (int)(t % NB);
  t /= NB;
  const int ks = (int)(t % KS);
  const long long lc = t / KS;
  const int n = nb * 32 + (lane & 31);
  const int k = ks * 16 + 8 * (lane >> 5);
  Wp[idx] = *reinterpret_cast<const uint4*>(A + ((lc * d_r + n) * (long long)d_in + k));
}

__global__ __launch_bounds__(256) void copy_f32_kernel(const float4* A, float4* Wp, long long n4) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  if (idx < n4) Wp[idx] = A[idx];
}

// ---------------------------------------------------------------------------
// Work decoding shared by both transfer kernels.  Work items run role-major,
// then layer, then sequence, then row tile, so the workgroups in flight at
// any time share one map A[l, c] (kept in L2) and the two sender layers it
// reads, and consecutive receiver layers reuse a sender layer.
// ---------------------------------------------------------------------------
struct Item {
  int c, l, b, tile;
};

__device__ __forceinline__ Item decode_item(const TransferArgs& p, int item) {
  Item it;
  const int lc = item / p.tiles_per_lc;
  int t = item - lc * p.tiles_per_lc;
  it.c = lc / p.L_r;
  it.l = lc - it.c * p.L_r;
  int b = 0;
  while (b + 1 < p.B && p.tile_start[b + 1] <= t) ++b;
  it.b = b;
  it.tile = t - p.tile_start[b];
  return it;
}

// ---------------------------------------------------------------------------
// bf16 transfer kernel (d_h = 128).
//
// One workgroup = 8 waves computes MT = 64*WM receiver rows x all d_r = 128*WN
// receiver features of one (layer, role).  Wave (wm, wn) owns rows
// [64 wm, 64 wm + 64) and receiver head wn.  The contraction over the sender
// features runs one sender head (128 features) at a time:
//   build:  all 512 threads form the fp32 aligned/interpolated/un-rotated
//           features X[MT][128] of that head and store them as bf16 in LDS;
//   mma:    each wave multiplies its 128 x 64 (features x rows) output block
//           by that X slice on the matrix cores (operands: packed maps from
//           global memory as the A operand, X from LDS as the B operand).
// X is built once per row tile and reused for every output feature.  The
// accumulator of lane l, tile (mt, nt), register i holds receiver row
// 32 mt + l%32 and feature 32 nt + 8 (i/4) + 4 (l/32) + i%4 of the head, so
// a RoPE pair (f, f + 64) sits in tiles nt and nt + 2 of the same lane.
// The epilogue adds the bias, rotates keys, rounds to bf16 and writes through
// a per-wave LDS staging area so each global store covers whole 256-byte rows.
// ---------------------------------------------------------------------------
constexpr int kDH = 128;
constexpr int kXS = kDH + 8;  // LDS row stride in bf16 elements (16-byte pad)

template <int WN>
__global__ __launch_bounds__(512, 1) void transfer_bf16_kernel(const TransferArgs p) {
  constexpr int WM = 8 / WN;
  constexpr int MT = 64 * WM;
  constexpr int XBUF = MT * kXS;           // one X buffer, bf16 elements
  constexpr int STAGE = 32 * kXS;          // one wave's epilogue staging, bf16 elements
  constexpr int LDS = (2 * XBUF > 8 * STAGE) ? 2 * XBUF : 8 * STAGE;
  __shared__ __attribute__((aligned(16))) uint16_t lds[LDS];

  const Item it = decode_item(p, blockIdx.x);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int j0 = it.tile * MT;
  const int Tr = p.Tr[it.b], Ts = p.Ts[it.b];
  const int row0 = p.row0[it.b];
  const bool keys = it.c == 0;
  const bool unrot = keys && p.unrot;
  const bool rot = keys && p.rot;
  const float wlo = p.wlo[it.l], whi = p.whi[it.l];
  const bool two_tap = whi != 0.0f;
  const uint16_t* Sb = static_cast<const uint16_t*>(p.S) + it.b * p.s_sb + it.c * p.s_sc;
  const uint16_t* S_lo = Sb + (long long)p.lo[it.l] * p.s_sl;
  const uint16_t* S_hi = Sb + (long long)p.hi[it.l] * p.s_sl;
  const float2* cs_s = unrot ? p.cs_s + (long long)p.pos0_s[it.b] * (kDH / 2) : nullptr;

  const int KS = p.H_s * (kDH / 16);  // 16-wide k steps over all sender features
  const int NB = p.H_r * (kDH / 32);  // 32-row fragments over all receiver features
  const int lc_store = it.l * 2 + it.c;
  const bf16x8* W = static_cast<const bf16x8*>(p.Wp) + (long long)lc_store * KS * NB * 64;

  // Build mapping: 8 threads per row, thread owns features e0..e0+7 and
  // e0+64..e0+71 of the current sender head (a RoPE pair per index).
  const int brow = tid >> 3;
  const int e0 = (tid & 7) * 8;

  f32x16 acc[2][4];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[mt][nt][i] = 0.0f;

  for (int h = 0; h < p.H_s; ++h) {
    uint16_t* xb = lds + (h & 1) * XBUF;
    // ---- build X for sender head h ----
#pragma unroll
    for (int q = 0; q < WM; ++q) {
      const int r = brow + 64 * q;
      const int j = j0 + r;
      float x[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) x[u] = 0.0f;
      if (j < Tr) {
        const int g = row0 + j;
        const int e_beg = p.row_ptr[g], e_end = p.row_ptr[g + 1];
        const float dinv = (float)p.den[g];
        for (int e = e_beg; e < e_end; ++e) {
          int i = p.col[e];
          i = min(max(i, 0), Ts - 1);
          const float w = (float)p.num[e] / dinv;
          const long long off = h * p.s_sh + (long long)i * p.s_st + e0;
          float m[16], t[16];
          unpack8(*reinterpret_cast<const uint4*>(S_lo + off), m);
          unpack8(*reinterpret_cast<const uint4*>(S_lo + off + 64), m + 8);
#pragma unroll
          for (int u = 0; u < 16; ++u) m[u] *= wlo;
          if (two_tap) {
            unpack8(*reinterpret_cast<const uint4*>(S_hi + off), t);
            unpack8(*reinterpret_cast<const uint4*>(S_hi + off + 64), t + 8);
#pragma unroll
            for (int u = 0; u < 16; ++u) m[u] = fmaf(whi, t[u], m[u]);
          }
          if (unrot) {
            const float4* cs = reinterpret_cast<const float4*>(cs_s + (long long)i * (kDH / 2) + e0);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const float4 v = cs[u];  // (cos, sin) of features e0+2u and e0+2u+1
              const float c0 = v.x, s0 = v.y, c1 = v.z, s1 = v.w;
              const float a0 = m[2 * u], b0 = m[2 * u + 8], a1 = m[2 * u + 1], b1 = m[2 * u + 9];
              m[2 * u] = fmaf(a0, c0, b0 * s0);
              m[2 * u + 8] = fmaf(b0, c0, -a0 * s0);
              m[2 * u + 1] = fmaf(a1, c1, b1 * s1);
              m[2 * u + 9] = fmaf(b1, c1, -a1 * s1);
            }
          }
#pragma unroll
          for (int u = 0; u < 16; ++u) x[u] = fmaf(w, m[u], x[u]);
        }
      }
      *reinterpret_cast<uint4*>(xb + r * kXS + e0) = pack8(x);
      *reinterpret_cast<uint4*>(xb + r * kXS + e0 + 64) = pack8(x + 8);
    }
    __syncthreads();
    // ---- multiply: 8 k-steps of 16 over this head ----
    const bf16x8* Wh = W + (long long)h * 8 * NB * 64 + (wn * 4) * 64 + lane;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      bf16x8 xa[2], wf[4];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
        xa[mt] = *reinterpret_cast<const bf16x8*>(
            xb + (64 * wm + 32 * mt + (lane & 31)) * kXS + 16 * s + 8 * (lane >> 5));
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) wf[nt] = Wh[(s * NB + nt) * 64];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[nt], xa[mt], acc[mt][nt], 0, 0, 0);
    }
  }
  __syncthreads();  // every wave is done reading X; LDS becomes staging space

  // ---- epilogue ----
  const int hi4 = 4 * (lane >> 5);
  const int mcol = lane & 31;
  float bias_v[4][4][4];  // [nt][g][u]: feature 32 nt + 8 g + hi4 + u
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float4 bv = make_float4(0.f, 0.f, 0.f, 0.f);
      if (p.bias)
        bv = *reinterpret_cast<const float4*>(p.bias + (long long)lc_store * NB * 32 + wn * kDH +
                                              32 * nt + 8 * g + hi4);
      bias_v[nt][g][0] = bv.x; bias_v[nt][g][1] = bv.y;
      bias_v[nt][g][2] = bv.z; bias_v[nt][g][3] = bv.w;
    }
  uint16_t* stage = lds + wave * STAGE;
  uint16_t* Rb = static_cast<uint16_t*>(p.R) + it.b * p.r_sb + (long long)it.l * p.r_sl +
                 it.c * p.r_sc + wn * p.r_sh;
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
    const int rloc = 64 * wm + 32 * mt + mcol;  // row within the tile held by this lane
    const int j = j0 + rloc;
    float y[4][16];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int i = 0; i < 16; ++i) y[nt][i] = acc[mt][nt][i] + bias_v[nt][i >> 2][i & 3];
    if (rot && j < Tr) {
      const float2* cr = p.cs_r + (long long)(p.pos0_r[it.b] + j) * (kDH / 2);
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const float4* cp = reinterpret_cast<const float4*>(cr + 32 * nt + 8 * g + hi4);
          const float4 v0 = cp[0], v1 = cp[1];
          const float cc[4] = {v0.x, v0.z, v1.x, v1.z};
          const float ss[4] = {v0.y, v0.w, v1.y, v1.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float a = y[nt][4 * g + u], bq = y[nt + 2][4 * g + u];
            y[nt][4 * g + u] = fmaf(a, cc[u], -bq * ss[u]);
            y[nt + 2][4 * g + u] = fmaf(bq, cc[u], a * ss[u]);
          }
        }
    }
    // stage: row mcol, features 32 nt + 8 g + hi4 .. +3
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint2 v = make_uint2(pack2(y[nt][4 * g], y[nt][4 * g + 1]),
                             pack2(y[nt][4 * g + 2], y[nt][4 * g + 3]));
        *reinterpret_cast<uint2*>(stage + mcol * kXS + 32 * nt + 8 * g + hi4) = v;
      }
    // write back 32 rows x 256 bytes: 16 lanes per row, 4 rows per pass
#pragma unroll
    for (int pass = 0; pass < 8; ++pass) {
      const int rr = pass * 4 + (lane >> 4);
      const int cc = (lane & 15) * 8;
      const uint4 v = *reinterpret_cast<const uint4*>(stage + rr * kXS + cc);
      const int jj = j0 + 64 * wm + 32 * mt + rr;
      if (jj < Tr) *reinterpret_cast<uint4*>(Rb + (long long)jj * p.r_st + cc) = v;
    }
  }
}

// ---------------------------------------------------------------------------
// fp32 transfer kernel: the same definitions with fp32 operands and plain
// FMA, any even d_h.  One workgroup = RT receiver rows of one (layer, role).
// ---------------------------------------------------------------------------
constexpr int kF32Threads = 256;

__global__ __launch_bounds__(kF32Threads) void transfer_f32_kernel(const TransferArgs p) {
  extern __shared__ float xs[];  // [RT][d_in]
  const Item it = decode_item(p, blockIdx.x);
  const int RT = p.rows_per_tile;
  const int d = p.d_h, half = d / 2;
  const int d_in = p.H_s * d, d_r = p.H_r * d;
  const int j0 = it.tile * RT;
  const int Tr = p.Tr[it.b], Ts = p.Ts[it.b];
  const bool keys = it.c == 0;
  const bool unrot = keys && p.unrot, rot = keys && p.rot;
  const float wlo = p.wlo[it.l], whi = p.whi[it.l];
  const bool two_tap = whi != 0.0f;
  const float* Sb = static_cast<const float*>(p.S) + it.b * p.s_sb + it.c * p.s_sc;
  const float* S_lo = Sb + (long long)p.lo[it.l] * p.s_sl;
  const float* S_hi = Sb + (long long)p.hi[it.l] * p.s_sl;
  const int lc_store = it.l * 2 + it.c;

  for (int idx = threadIdx.x; idx < RT * p.H_s * half; idx += kF32Threads) {
    const int r = idx / (p.H_s * half);
    const int rem = idx - r * (p.H_s * half);
    const int h = rem / half, f = rem - h * half;
    const int j = j0 + r;
    float x1 = 0.f, x2 = 0.f;
    if (j < Tr) {
      const int g = p.row0[it.b] + j;
      const float dinv = (float)p.den[g];
      for (int e = p.row_ptr[g]; e < p.row_ptr[g + 1]; ++e) {
        int i = min(max(p.col[e], 0), Ts - 1);
        const float w = (float)p.num[e] / dinv;
        const long long off = h * p.s_sh + (long long)i * p.s_st + f;
        float m1 = wlo * S_lo[off], m2 = wlo * S_lo[off + half];
        if (two_tap) {
          m1 = fmaf(whi, S_hi[off], m1);
          m2 = fmaf(whi, S_hi[off + half], m2);
        }
        if (unrot) {
          const float2 cs = p.cs_s[(long long)(p.pos0_s[it.b] + i) * half + f];
          const float u1 = fmaf(m1, cs.x, m2 * cs.y);
          const float u2 = fmaf(m2, cs.x, -m1 * cs.y);
          m1 = u1;
          m2 = u2;
        }
        x1 = fmaf(w, m1, x1);
        x2 = fmaf(w, m2, x2);
      }
    }
    xs[r * d_in + h * d + f] = x1;
    xs[r * d_in + h * d + f + half] = x2;
  }
  __syncthreads();

  const float* W = static_cast<const float*>(p.Wp) + (long long)lc_store * d_r * d_in;
  float* Rb = static_cast<float*>(p.R) + it.b * p.r_sb + (long long)it.l * p.r_sl + it.c * p.r_sc;
  constexpr int kMaxRT = 16;
  for (int pc = threadIdx.x; pc < p.H_r * half; pc += kF32Threads) {
    const int hr = pc / half, f = pc - hr * half;
    const int n1 = hr * d + f, n2 = n1 + half;
    float y1[kMaxRT], y2[kMaxRT];
#pragma unroll
    for (int r = 0; r < kMaxRT; ++r) y1[r] = y2[r] = 0.f;
    const float* W1 = W + (long long)n1 * d_in;
    const float* W2 = W + (long long)n2 * d_in;
    for (int k = 0; k < d_in; ++k) {
      const float a1 = W1[k], a2 = W2[k];
#pragma unroll
      for (int r = 0; r < kMaxRT; ++r) {
        if (r < RT) {
          const float xv = xs[r * d_in + k];
          y1[r] = fmaf(a1, xv, y1[r]);
          y2[r] = fmaf(a2, xv, y2[r]);
        }
      }
    }
    const float b1 = p.bias ? p.bias[(long long)lc_store * d_r + n1] : 0.f;
    const float b2 = p.bias ? p.bias[(long long)lc_store * d_r + n2] : 0.f;
#pragma unroll
    for (int r = 0; r < kMaxRT; ++r) {
      const int j = j0 + r;
      if (r >= RT || j >= Tr) continue;
      float v1 = y1[r] + b1, v2 = y2[r] + b2;
      if (rot) {
        const float2 cs = p.cs_r[(long long)(p.pos0_r[it.b] + j) * half + f];
        const float u1 = fmaf(v1, cs.x, -v2 * cs.y);
        const float u2 = fmaf(v2, cs.x, v1 * cs.y);
        v1 = u1;
        v2 = u2;
      }
      float* dst = Rb + hr * p.r_sh + (long long)j * p.r_st;
      dst[f] = v1;
      dst[f + half] = v2;
    }
  }
}

}  // namespace

int transfer_rows_per_tile(int dtype, int H_r, int d_in) {
  if (dtype == HF_BF16) return 64 * (8 / (H_r > 0 ? H_r : 1));
  int rt = 8192 / (d_in > 0 ? d_in : 1);  // fp32 X tile <= 32 KB of LDS
  return rt < 1 ? 1 : (rt > 16 ? 16 : rt);
}

hipError_t launch_rope_table(float2* tab, int P, int d_h, double theta, hipStream_t s) {
  const int half = d_h / 2;
  const long long n = (long long)P * half;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, tab, P,
                     half, d_h, theta);
  return hipGetLastError();
}

hipError_t launch_pack_maps(int dtype, int n_lc, int d_r, int d_in, const void* A, void* Wp,
                            hipStream_t s) {
  if (dtype == HF_BF16) {
    const long long n = (long long)n_lc * (d_r / 32) * (d_in / 16) * 64;
    if (n > 0)
      hipLaunchKernelGGL(pack_bf16_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                         static_cast<const uint16_t*>(A), static_cast<uint4*>(Wp), n, d_r, d_in);
  } else {
    const long long n4 = (long long)n_lc * d_r * d_in / 4;
    if (n4 > 0)
      hipLaunchKernelGGL(copy_f32_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s,
                         static_cast<const float4*>(A), static_cast<float4*>(Wp), n4);
  }
  return hipGetLastError();
}

hipError_t launch_transfer(int dtype, const TransferArgs& a, hipStream_t s) {
  const long long items = (long long)a.tiles_per_lc * a.L_r * 2;
  if (items <= 0) return hipSuccess;
  const dim3 grid((unsigned)items);
  if (dtype == HF_BF16) {
    switch (a.H_r) {
      case 2: hipLaunchKernelGGL(transfer_bf16_kernel<2>, grid, dim3(512), 0, s, a); break;
      case 4: hipLaunchKernelGGL(transfer_bf16_kernel<4>, grid, dim3(512), 0, s, a); break;
      case 8: hipLaunchKernelGGL(transfer_bf16_kernel<8>, grid, dim3(512), 0, s, a); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    const size_t shmem = (size_t)a.rows_per_tile * a.H_s * a.d_h * sizeof(float);
    hipLaunchKernelGGL(transfer_f32_kernel, grid, dim3(kF32Threads), shmem, s, a);
  }
  return hipGetLastError();
}

}  // namespace hf
