// KV transfer kernels: RoPE cos/sin tables, map packing, and the transfer
// itself (layer interpolation + RoPE un-rotation + overlap-weighted segment
// mean, then the folded affine map of Eq. 9 with bias and receiver RoPE in
// the epilogue, written straight into the receiver cache layout).
#include <hip/hip_runtime.h>

#include <cstddef>
#include <limits.h>

#include <mutex>
#include <type_traits>

#include "hf_internal.h"

namespace hf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;

// ---------------------------------------------------------------------------
// bf16 helpers.  bf16 -> f32 is exact (the bf16 bits are the top half of the
// f32); f32 -> bf16 rounds to nearest even (v_cvt_pk_bf16_f32).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

__device__ __forceinline__ uint32_t pack2(float a, float b) {
  bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint4 pack8(const float* f) {
  return make_uint4(pack2(f[0], f[1]), pack2(f[2], f[3]), pack2(f[4], f[5]), pack2(f[6], f[7]));
}

// One 16-byte-per-lane global -> LDS copy: lane l writes 16 bytes at
// lds_wave_base + 16 l (lds_wave_base must be the same for the whole wave).
__device__ __forceinline__ void copy16_to_lds(const void* gsrc, void* lds_wave_base) {
  __builtin_amdgcn_global_load_lds(gsrc, (lds_void_t*)lds_wave_base, 16, 0, 0);
}

// ---------------------------------------------------------------------------
// RoPE tables: row pos holds cos(pos w_k) for k < d/2, then sin(pos w_k), with
// w_k = theta^(-2k/d); the angle is formed in fp64.
// ---------------------------------------------------------------------------
// A thread owns one angle index k (threadIdx.x + 64 blockIdx.y) and kRopePpt
// consecutive positions, so w_k is formed once per thread.
constexpr int kRopePpt = 16;
__global__ __launch_bounds__(256) void rope_table_kernel(float* tab, int P, int half, int d,
                                                         double theta) {
  const int k = blockIdx.y * 64 + threadIdx.x;
  if (k >= half) return;
  const double w = pow(theta, -2.0 * k / d);
  const long long p0 = ((long long)blockIdx.x * 4 + threadIdx.y) * kRopePpt;
  const int p1 = (int)min(p0 + kRopePpt, (long long)P);
  for (int pos = (int)min(p0, (long long)P); pos < p1; ++pos) {
    double s, c;
    sincos((double)pos * w, &s, &c);
    tab[(long long)pos * d + k] = (float)c;
    tab[(long long)pos * d + half + k] = (float)s;
  }
}

// ---------------------------------------------------------------------------
// Map packing for the bf16 matrix-core kernels.  One 1 KB fragment holds the
// 32 x 16 block (rows n, columns k) one v_mfma_f32_32x32x16_bf16 consumes as
// its A operand: lane l holds row n = 32 nb + l%32, columns
// k = 16 ks + 8 (l/32) + 0..7.  Fragments are ordered [lc][ks][nb], so a wave
// reads one fragment with a single fully coalesced 16-byte-per-lane load.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void pack_bf16_kernel(const uint16_t* A, uint4* Wp,
                                                        long long n_frag_lanes, int d_r, int d_in) {
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

// Header of a packed map buffer: what hf_pack_maps packed, ahead of the data.
__global__ __launch_bounds__(64) void pack_header_kernel(uint32_t* hdr, int dtype, int L_r,
                                                         int d_r, int d_in) {
  const int i = threadIdx.x;
  uint32_t v = 0;
  if (i == 0) v = kPackedMagic;
  if (i == 1) v = 1;  // layout version
  if (i == 2) v = (uint32_t)dtype;
  if (i == 3) v = (uint32_t)L_r;
  if (i == 4) v = (uint32_t)d_r;
  if (i == 5) v = (uint32_t)d_in;
  hdr[i] = v;  // 64 words = HF_PACKED_HEADER_BYTES
}

__global__ __launch_bounds__(256) void copy_f32_kernel(const float4* A, float4* Wp, long long n4) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  if (idx < n4) Wp[idx] = A[idx];
}

// ---------------------------------------------------------------------------
// Work decoding shared by the transfer kernels.  Work items run role-major,
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

constexpr int kDH = 128;
constexpr int kXS = kDH + 8;  // LDS row stride of X / staging, bf16 elements (16-byte pad)

// Per-(layer, role, sequence) constants of the bf16 kernels.
struct Ctx {
  const uint16_t* S_lo;   // sender cache at (b, lo, c), head 0, token 0
  const uint16_t* S_hi;
  const float* cs_s;      // sender RoPE table row of position pos0_s (nullptr: no un-rotation)
  float wlo, whi;
  bool two_tap;
  int Ts;
};

// Byte i of a kernel-argument byte array (lo, hi, taps), read as the aligned
// dword that holds it with a uniform index: gfx950 has no scalar byte loads,
// and a vector load here would wait (in order) for every load and store the
// workgroup still has in flight, such as the previous tile's receiver rows.
static_assert(offsetof(TransferArgs, lo) % 4 == 0 && offsetof(TransferArgs, hi) % 4 == 0 &&
                  offsetof(TransferArgs, taps) % 4 == 0,
              "layer-map byte arrays must be dword aligned");
__device__ __forceinline__ int arg_byte(const uint8_t* base, int i) {
  i = __builtin_amdgcn_readfirstlane(i);
  const uint32_t w = reinterpret_cast<const uint32_t*>(base)[i >> 2];
  return (int)((w >> (8 * (i & 3))) & 0xffu);
}

// Tap t of the layer map: with concatenated taps, sender layer taps[l][t]
// with weight 1; otherwise (t = 0) the interpolation of lo and hi.
__device__ __forceinline__ Ctx make_ctx(const TransferArgs& p, const Item& it, int t = 0) {
  Ctx x;
  const uint16_t* Sb = static_cast<const uint16_t*>(p.S) + it.b * p.s_sb + it.c * p.s_sc;
  const int lo = p.concat ? arg_byte(&p.taps[0][0], 3 * it.l + t) : arg_byte(p.lo, it.l);
  x.S_lo = Sb + (long long)lo * p.s_sl;
  x.S_hi = Sb + (long long)(p.concat ? lo : arg_byte(p.hi, it.l)) * p.s_sl;
  x.cs_s = (it.c == 0 && p.unrot) ? p.cs_s + (long long)p.pos0_s[it.b] * kDH : nullptr;
  x.wlo = p.concat ? 1.0f : p.wlo[it.l];
  x.whi = p.concat ? 0.0f : p.whi[it.l];
  x.two_tap = x.whi != 0.0f;
  if (p.inv_r) {  // the map sees x / r: scale the layer weights
    const float s = p.inv_r[it.l * 2 + it.c];
    x.wlo *= s;
    x.whi *= s;
  }
  x.Ts = p.Ts[it.b];
  return x;
}

// Accumulate the aligned features of one receiver row straight from global
// memory: x[0..7] = features e0..e0+7 and x[8..15] = e0+64..e0+71 of sender
// head h (a RoPE pair per index).  Used where the staged path does not apply.
__device__ __forceinline__ void build_row_global(const TransferArgs& p, const Ctx& cx, int g,
                                                 int h, int e0, float* x) {
  const int e_beg = p.row_ptr[g], e_end = p.row_ptr[g + 1];
  const float dinv = (float)p.den[g];
  for (int e = e_beg; e < e_end; ++e) {
    const int i = min(max(p.col[e], 0), cx.Ts - 1);
    const float w = (float)p.num[e] / dinv;
    const long long off = h * p.s_sh + (long long)i * p.s_st + e0;
    const uint4 L0 = *reinterpret_cast<const uint4*>(cx.S_lo + off);
    const uint4 L1 = *reinterpret_cast<const uint4*>(cx.S_lo + off + 64);
    uint4 H0 = make_uint4(0, 0, 0, 0), H1 = H0;
    if (cx.two_tap) {
      H0 = *reinterpret_cast<const uint4*>(cx.S_hi + off);
      H1 = *reinterpret_cast<const uint4*>(cx.S_hi + off + 64);
    }
    const float a = w * cx.wlo, bq = w * cx.whi;
    const uint32_t l0[4] = {L0.x, L0.y, L0.z, L0.w}, l1[4] = {L1.x, L1.y, L1.z, L1.w};
    const uint32_t h0[4] = {H0.x, H0.y, H0.z, H0.w}, h1[4] = {H1.x, H1.y, H1.z, H1.w};
    float cc[8], ss[8];
    if (cx.cs_s) {
      const float* row = cx.cs_s + (long long)i * kDH;
      const float4 c0 = *reinterpret_cast<const float4*>(row + e0);
      const float4 c1 = *reinterpret_cast<const float4*>(row + e0 + 4);
      const float4 s0 = *reinterpret_cast<const float4*>(row + 64 + e0);
      const float4 s1 = *reinterpret_cast<const float4*>(row + 64 + e0 + 4);
      cc[0] = c0.x; cc[1] = c0.y; cc[2] = c0.z; cc[3] = c0.w;
      cc[4] = c1.x; cc[5] = c1.y; cc[6] = c1.z; cc[7] = c1.w;
      ss[0] = s0.x; ss[1] = s0.y; ss[2] = s0.z; ss[3] = s0.w;
      ss[4] = s1.x; ss[5] = s1.y; ss[6] = s1.z; ss[7] = s1.w;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      float ma = a * ((u & 1) ? bf_hi(l0[u >> 1]) : bf_lo(l0[u >> 1]));
      float mb = a * ((u & 1) ? bf_hi(l1[u >> 1]) : bf_lo(l1[u >> 1]));
      if (cx.two_tap) {
        ma = fmaf(bq, (u & 1) ? bf_hi(h0[u >> 1]) : bf_lo(h0[u >> 1]), ma);
        mb = fmaf(bq, (u & 1) ? bf_hi(h1[u >> 1]) : bf_lo(h1[u >> 1]), mb);
      }
      if (cx.cs_s) {  // U(p) = R(-p) on the pair (e0 + u, e0 + 64 + u)
        x[u] = fmaf(ma, cc[u], fmaf(mb, ss[u], x[u]));
        x[u + 8] = fmaf(mb, cc[u], fmaf(-ma, ss[u], x[u + 8]));
      } else {
        x[u] += ma;
        x[u + 8] += mb;
      }
    }
  }
}

// 1 / sqrt(mean(y^2) + eps) of one receiver head row of 128 features whose
// squares are split between this lane (ss) and lane ^ 32.
__device__ __forceinline__ float rms_scale_pair(float ss, float eps) {
  ss += __shfl_xor(ss, 32);
  return 1.0f / sqrtf(ss * (1.0f / kDH) + eps);
}

// y[q][4 g + u] *= inv * weight of its feature feat[q] + 8 g + hi4 + u.
template <int NTW>
__device__ __forceinline__ void scale_by_weights(float (*y)[16], const int* feat, int hi4,
                                                 const float* wrow, float inv) {
#pragma unroll
  for (int q = 0; q < NTW; ++q)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const float4 w = *reinterpret_cast<const float4*>(wrow + feat[q] + 8 * g + hi4);
      y[q][4 * g + 0] *= inv * w.x;
      y[q][4 * g + 1] *= inv * w.y;
      y[q][4 * g + 2] *= inv * w.z;
      y[q][4 * g + 3] *= inv * w.w;
    }
}

// Epilogue of one 32-row block of a wave: bias, receiver RoPE on keys, bf16
// rounding, then a write through the wave's LDS staging rows so that global
// stores cover whole contiguous row segments.
//   acc[q]  accumulators of the wave's n-tile q (NTW of them) for these rows;
//   feat[q] first feature (within the receiver head) of n-tile q;
//   tiles q and q + NTW/2 hold the RoPE pair (f, f + 64).
template <int NTW>
__device__ __forceinline__ void epilogue_rows(const TransferArgs& p, f32x16* acc, const int* feat,
                                              const float* bias_head, const float* cr, bool rot,
                                              const float* knorm, uint16_t* stage,
                                              uint16_t* dst_head, int row_base, int Tr, int lane) {
  static_assert(NTW == 4, "the key norm needs the whole head in the wave");
  const int hi4 = 4 * (lane >> 5);
  const int mcol = lane & 31;
  const int j = row_base + mcol;
  float y[NTW][16];
#pragma unroll
  for (int q = 0; q < NTW; ++q)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float4 bv = make_float4(0.f, 0.f, 0.f, 0.f);
      if (bias_head) bv = *reinterpret_cast<const float4*>(bias_head + feat[q] + 8 * g + hi4);
      y[q][4 * g + 0] = acc[q][4 * g + 0] + bv.x;
      y[q][4 * g + 1] = acc[q][4 * g + 1] + bv.y;
      y[q][4 * g + 2] = acc[q][4 * g + 2] + bv.z;
      y[q][4 * g + 3] = acc[q][4 * g + 3] + bv.w;
    }
  if (knorm) {  // receiver key RMSNorm over the head's 128 features (lanes l, l ^ 32)
    float ss = 0.0f;
#pragma unroll
    for (int q = 0; q < NTW; ++q)
#pragma unroll
      for (int i = 0; i < 16; ++i) ss = fmaf(y[q][i], y[q][i], ss);
    scale_by_weights<NTW>(y, feat, hi4, knorm, rms_scale_pair(ss, p.k_norm_eps));
  }
  if (rot && j < Tr) {
    const float* crow = cr + (long long)j * kDH;
#pragma unroll
    for (int q = 0; q < NTW / 2; ++q)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int f = feat[q] + 8 * g + hi4;  // < 64
        const float4 cv = *reinterpret_cast<const float4*>(crow + f);
        const float4 sv = *reinterpret_cast<const float4*>(crow + 64 + f);
        const float cc[4] = {cv.x, cv.y, cv.z, cv.w};
        const float ss[4] = {sv.x, sv.y, sv.z, sv.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float a = y[q][4 * g + u], b = y[q + NTW / 2][4 * g + u];
          y[q][4 * g + u] = fmaf(a, cc[u], -b * ss[u]);
          y[q + NTW / 2][4 * g + u] = fmaf(b, cc[u], a * ss[u]);
        }
      }
  }
  // stage row mcol: tile q occupies staging columns [32 q, 32 q + 32)
#pragma unroll
  for (int q = 0; q < NTW; ++q)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint2 v = make_uint2(pack2(y[q][4 * g], y[q][4 * g + 1]), pack2(y[q][4 * g + 2], y[q][4 * g + 3]));
      *reinterpret_cast<uint2*>(stage + mcol * kXS + 32 * q + 8 * g + hi4) = v;
    }
  // write back: NTW*4 lanes per row, each 16 bytes
  constexpr int LPR = NTW * 4;
  constexpr int RPP = 64 / LPR;
#pragma unroll
  for (int pass = 0; pass < 32 / RPP; ++pass) {
    const int rr = pass * RPP + lane / LPR;
    const int ci = lane % LPR;
    const uint4 v = *reinterpret_cast<const uint4*>(stage + rr * kXS + 8 * ci);
    const int jj = row_base + rr;
    if (jj < Tr)
      *reinterpret_cast<uint4*>(dst_head + (long long)jj * p.r_st + feat[ci / 4] + 8 * (ci % 4)) = v;
  }
}

// ---------------------------------------------------------------------------
// bf16 transfer kernel, tiled (d_h = 128, up to 8 sender heads; NTW = 4 for 8
// receiver heads, NTW = 2 for 4).
//
// One workgroup = 8 waves computes 64 receiver rows x all d_r receiver
// features of one (layer, role), in three phases after copying the tile's
// staging record (stage_tiles_kernel) into LDS:
//   build: all 512 threads form the whole aligned feature block X[64][d_in]
//          in fp32 -- gather the tile's CSR entries (from the record), mix the
//          two sender-layer taps, un-rotate keys, weight and sum -- and store
//          it once as bf16 in LDS.  Sender rows come straight from global
//          memory through a register ring of trips; no matrix-core work is in
//          flight, so nothing waits behind these loads.  Each lane group walks
//          a run of rows holding an equal share of the tile's entries.
//   mma:   each wave multiplies its output tiles by X over all d_in/16 k-steps
//          (v_mfma_f32_32x32x16_bf16: packed map fragment from global memory as
//          A, X from LDS as B) with a four-deep register prefetch of the map
//          fragments and no barrier inside the loop.  Workgroups start the loop
//          at different sender heads so that concurrent workgroups stream
//          different parts of the map.
//   store: the tile's receiver RoPE rows and the bias are copied into LDS
//          once; bias, rotation and bf16 rounding, then staged row writes.
// Wave w owns NTW 32-feature tiles of one receiver head (NTW = 4: the whole
// head w; NTW = 2: tiles {w%2, w%2 + 2} of head w/2), so RoPE pairs
// (f, f + 64) stay inside a lane; the accumulator of lane l, row block mt,
// tile q, register i holds receiver row 32 mt + l%32 and feature
// feat[q] + 8 (i/4) + 4 (l/32) + i%4.
//
// The un-rotation of sender row i at position p_i is split as
// U(p_i) = U(q_g) U(p_i - q_g) with q_g the position of the smallest sender
// token of the lane group's run: the small-offset rotations U(0..15) sit in
// LDS and U(q_g) is applied once to each row's sum.  Tiles whose entry count or
// run sender span exceed what is staged build X entry by entry from the CSR
// and the full RoPE table in global memory (same results).
// ---------------------------------------------------------------------------
constexpr int kEMax = 512;             // CSR entries staged per tile
constexpr int kDMax = kRopeDeltaRows;  // in-row sender offsets handled with the LDS table
constexpr int kHMax = 8;               // sender heads held in LDS
constexpr int kXF = kHMax * kDH + 8;   // LDS row stride of X, bf16 elements (16-byte pad)
constexpr int kXBytes = 64 * kXF * 2;
constexpr int kDtBytes = kDMax * kDH * 4;            // U(delta) rows: cos | sin, fp32
constexpr int kOffDt = kXBytes;
constexpr int kOffEnt = kOffDt + kDtBytes;
// Staged tile record: estart, gbase, ecol, ew, einfo, flags, gstart, row min /
// max sender index; written once per row tile by the staging kernel and copied
// whole into LDS by every (layer, role) of the tile.
constexpr int kEntInts = 65 + 64 + kEMax * 3 + 4 + 65 + 2 * 64;
constexpr int kRecBytes = 8192;  // 8 waves x 64 lanes x 16 bytes
static_assert(kEntInts * 4 <= kRecBytes, "tile record size");
constexpr int kOffNext = kOffEnt + kRecBytes;  // the workgroup's next work item
constexpr int kSmemBytes = kOffNext + 16;
// Store phase, inside the (then free) X region: receiver RoPE rows, bias, staging.
constexpr int kOffRcs = 0;                           // [64][cos 64 | sin 64] fp32
constexpr int kOffBias = kOffRcs + 64 * kDH * 4;     // [d_r <= 1024] fp32
constexpr int kOffStage = kOffBias + 1024 * 4;       // 8 waves x [32][kXS] bf16
constexpr int kOffRsum = kOffStage + 8 * 32 * kXS * 2;  // 8 waves x 32 fp32
static_assert(kOffRsum + 8 * 32 * 4 <= kXBytes, "store phase must fit the X region");
static_assert(kSmemBytes <= 160 * 1024, "LDS budget");

// Group-walk build.  WPH waves share a sender head, 8 WPH lane groups (8
// lanes, 16 features each) over the tile's 64 rows: group g walks the CSR
// entries of a run of consecutive rows in order, one entry per trip, so a
// sender token shared by neighbouring rows is read twice in a row (the second
// read hits the cache).  The runs hold equal shares of the tile's entries, as
// a wave takes as many trips as its longest run.  Trips past a group's last entry
// use an out-of-range buffer offset, which returns zeros without touching
// memory, so every trip issues the same loads and a ring of R trips keeps
// R - 1 trips of loads in flight.
constexpr int kOOB = (int)0x80000000;  // buffer offset past any slab extent (extents < 2^31)

struct GroupLds {
  const int* estart;  // [65] CSR offsets of the tile rows
  const int* ecol;    // staged sender indices
  const float* ew;    // staged weights num / den
  const int* einfo;   // staged row | last-entry-of-row << 8 | first-entry-of-row << 9
  const float* dt;    // U(0..15), swizzled
  int e_base;
};

template <bool TWO_TAP>
struct Trip {
  uint4 a0, a1, b0, b1;  // tap lo / hi: features e0..e0+7 and e0+64..e0+71
  int code;              // -1: no entry; else row | last << 6 | (i - base) << 8
  float w;
};

// Rotation rows of the swizzled U(0..15) table: row t holds cos chunks 0..15
// then sin chunks 16..31 (4 floats each), chunk c stored at slot c ^ (t & 1).
__device__ __forceinline__ void table_row(const float* tab, int t, int e0, float* c, float* s) {
  const float4* row = reinterpret_cast<const float4*>(tab) + t * 32;
  const int cw = t & 1;
  const float4 c0 = row[(e0 >> 2) ^ cw], c1 = row[((e0 >> 2) + 1) ^ cw];
  const float4 s0 = row[(16 + (e0 >> 2)) ^ cw], s1 = row[(17 + (e0 >> 2)) ^ cw];
  c[0] = c0.x; c[1] = c0.y; c[2] = c0.z; c[3] = c0.w;
  c[4] = c1.x; c[5] = c1.y; c[6] = c1.z; c[7] = c1.w;
  s[0] = s0.x; s[1] = s0.y; s[2] = s0.z; s[3] = s0.w;
  s[4] = s1.x; s[5] = s1.y; s[6] = s1.z; s[7] = s1.w;
}

__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, int off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// Where a built X row goes: sink(r, f, v) stores features f..f+7 of tile row r.
struct LdsSink {  // the X tile in LDS (row stride kXF)
  uint16_t* Xs;
  __device__ __forceinline__ void operator()(int r, int f, uint4 v) const {
    *reinterpret_cast<uint4*>(Xs + r * kXF + f) = v;
  }
};

template <bool TWO_TAP, bool UNROT, int R, class Sink>
__device__ __forceinline__ void build_groups(const Ctx& cx, const TransferArgs& p, const GroupLds& L,
                                             int base, int head, int r_first, int rpg, int lane,
                                             const Sink& sink) {
  const int e0 = (lane & 7) * 8;
  const int kb = L.estart[r_first] - L.e_base;
  const int E = L.estart[r_first + rpg] - L.e_base - kb;
  int T = 0;  // trips of the wave: the longest group
#pragma unroll
  for (int g = 0; g < 8; ++g) T = max(T, __builtin_amdgcn_readlane(E, 8 * g));
  for (int q = 0; q < rpg; ++q) {  // rows without entries stay zero
    const int r = r_first + q;
    if (L.estart[r + 1] == L.estart[r]) {
      sink(r, head * kDH + e0, make_uint4(0, 0, 0, 0));
      sink(r, head * kDH + 64 + e0, make_uint4(0, 0, 0, 0));
    }
  }
  float rc[8], rs[8];  // U(p_base): closes every row of the group
  if (UNROT) {
    const float* row = cx.cs_s + (long long)base * kDH;
    const float4 c0 = *reinterpret_cast<const float4*>(row + e0);
    const float4 c1 = *reinterpret_cast<const float4*>(row + e0 + 4);
    const float4 s0 = *reinterpret_cast<const float4*>(row + 64 + e0);
    const float4 s1 = *reinterpret_cast<const float4*>(row + 64 + e0 + 4);
    rc[0] = c0.x; rc[1] = c0.y; rc[2] = c0.z; rc[3] = c0.w;
    rc[4] = c1.x; rc[5] = c1.y; rc[6] = c1.z; rc[7] = c1.w;
    rs[0] = s0.x; rs[1] = s0.y; rs[2] = s0.z; rs[3] = s0.w;
    rs[4] = s1.x; rs[5] = s1.y; rs[6] = s1.z; rs[7] = s1.w;
  }
  const __amdgpu_buffer_rsrc_t rlo =
      __builtin_amdgcn_make_buffer_rsrc((void*)cx.S_lo, 0, p.s_extent, 0x00020000);
  const __amdgpu_buffer_rsrc_t rhi =
      __builtin_amdgcn_make_buffer_rsrc((void*)cx.S_hi, 0, p.s_extent, 0x00020000);
  const int hoff = (int)(head * p.s_sh + e0) * 2;  // bytes
  const int tstride = (int)p.s_st * 2;

  Trip<TWO_TAP> ring[R];
  float x[16];
#pragma unroll
  for (int u = 0; u < 16; ++u) x[u] = 0.0f;

  auto issue = [&](Trip<TWO_TAP>& t, int k) {
    const bool valid = k < E;
    int i = 0, info = 0;
    float w = 0.0f;
    if (valid) {
      i = L.ecol[kb + k];
      w = L.ew[kb + k];
      info = L.einfo[kb + k];
    }
    const int off = valid ? hoff + i * tstride : kOOB;
    t.a0 = buf_load16(rlo, off);
    t.a1 = buf_load16(rlo, off + 128);
    if (TWO_TAP) {
      t.b0 = buf_load16(rhi, off);
      t.b1 = buf_load16(rhi, off + 128);
    }
    t.code = valid ? ((info & 63) | ((info >> 8) << 6) | ((UNROT ? i - base : 0) << 8)) : -1;
    t.w = w;
  };
  auto consume = [&](const Trip<TWO_TAP>& t) {
    if (t.code < 0) return;
    const uint32_t l0[4] = {t.a0.x, t.a0.y, t.a0.z, t.a0.w};
    const uint32_t l1[4] = {t.a1.x, t.a1.y, t.a1.z, t.a1.w};
    uint32_t h0[4] = {0, 0, 0, 0}, h1[4] = {0, 0, 0, 0};
    if (TWO_TAP) {
      h0[0] = t.b0.x; h0[1] = t.b0.y; h0[2] = t.b0.z; h0[3] = t.b0.w;
      h1[0] = t.b1.x; h1[1] = t.b1.y; h1[2] = t.b1.z; h1[3] = t.b1.w;
    }
    const float a = t.w * cx.wlo, bq = t.w * cx.whi;  // weight folded into the layer mix
    float cc[8], ss[8];
    if (UNROT) table_row(L.dt, t.code >> 8, e0, cc, ss);  // U(p_i - p_base)
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      float ma = a * ((u & 1) ? bf_hi(l0[u >> 1]) : bf_lo(l0[u >> 1]));
      float mb = a * ((u & 1) ? bf_hi(l1[u >> 1]) : bf_lo(l1[u >> 1]));
      if (TWO_TAP) {
        ma = fmaf(bq, (u & 1) ? bf_hi(h0[u >> 1]) : bf_lo(h0[u >> 1]), ma);
        mb = fmaf(bq, (u & 1) ? bf_hi(h1[u >> 1]) : bf_lo(h1[u >> 1]), mb);
      }
      if (UNROT) {
        x[u] = fmaf(ma, cc[u], fmaf(mb, ss[u], x[u]));
        x[u + 8] = fmaf(mb, cc[u], fmaf(-ma, ss[u], x[u + 8]));
      } else {
        x[u] += ma;
        x[u + 8] += mb;
      }
    }
    if ((t.code >> 6) & 1) {  // last entry of the row: close the rotation, round, store
      if (UNROT) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const float a = x[u], b = x[u + 8];
          x[u] = fmaf(a, rc[u], b * rs[u]);
          x[u + 8] = fmaf(b, rc[u], -a * rs[u]);
        }
      }
      sink(t.code & 63, head * kDH + e0, pack8(x));
      sink(t.code & 63, head * kDH + 64 + e0, pack8(x + 8));
#pragma unroll
      for (int u = 0; u < 16; ++u) x[u] = 0.0f;
    }
  };

#pragma unroll
  for (int s = 0; s < R - 1; ++s) issue(ring[s], s);
  for (int t0 = 0; t0 < T; t0 += R) {
#pragma unroll
    for (int s = 0; s < R; ++s) {
      issue(ring[(s + R - 1) % R], t0 + s + R - 1);
      if (t0 + s < T) consume(ring[s]);
    }
  }
}

// ---------------------------------------------------------------------------
// Per-tile staging for the tiled kernel, one workgroup per 64-row tile of the
// batch.  The record holds the tile's CSR entries with their row, weight
// num/den and first / last-of-row flags; the cut of the rows into runs of
// consecutive rows with equal shares of the entries (a wave takes as many
// trips as its longest run); each run's smallest sender index; and two flags:
// [0] some run spans kDMax sender tokens or more (too wide for the LDS
// rotation table), [1] the tile has more than kEMax entries.  Every (layer,
// role) of the tile reads the same record.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(512) void stage_tiles_kernel(const TransferArgs p, int* rec) {
  if (blockIdx.x == 0 && threadIdx.x == 0) *p.work_ctr = p.n_wg;  // items [0, n_wg) start statically
  __shared__ __attribute__((aligned(16))) int ent[kRecBytes / 4];
  int* estart = ent;
  int* gbase = estart + 65;
  int* ecol = gbase + 64;
  float* ew = reinterpret_cast<float*>(ecol + kEMax);
  int* einfo = reinterpret_cast<int*>(ew + kEMax);
  int* flag = einfo + kEMax;
  int* gstart = flag + 4;     // lane group g walks tile rows [gstart[g], gstart[g + 1])
  int* rmin = gstart + 65;    // smallest / largest sender index of each tile row
  int* rmax = rmin + 64;

  const int t = blockIdx.x;
  int b = 0;
  while (b + 1 < p.B && p.tile_start[b + 1] <= t) ++b;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int j0 = (t - p.tile_start[b]) * 64;
  const int nrows = min(64, p.Tr[b] - j0);
  const int g0 = p.row0[b] + j0;
  const int Ts = p.Ts[b];
  const int H = p.H_s;
  const int WPH = H == 1 ? 8 : H == 2 ? 4 : H <= 4 ? 2 : 1;  // waves per sender head

  if (tid <= 64) estart[tid] = p.row_ptr[g0 + min(tid, nrows)];
  if (tid < 4) flag[tid] = 0;
  __syncthreads();
  const int e_base = estart[0];
  const int nnz = estart[nrows] - e_base;
  const bool fits = nnz <= kEMax;
  if (fits) {
    for (int k = tid; k < nnz; k += 512) {
      int lo = 0, hi = nrows;  // row r with estart[r] <= e_base + k < estart[r + 1]
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (estart[mid] <= e_base + k) lo = mid; else hi = mid;
      }
      const int e = e_base + k;
      ecol[k] = min(max(p.col[e], 0), Ts - 1);
      ew[k] = (float)p.num[e] / (float)p.den[g0 + lo];
      einfo[k] = lo | ((int)(e + 1 == estart[lo + 1]) << 8) | ((int)(e == estart[lo]) << 9);
    }
  }
  __syncthreads();
  const int NG = 8 * WPH;  // lane groups over the tile's rows
  if (wave == 0) {
    // Boundaries gstart[0..NG]; with one sender head NG = 64, one more than the
    // wave has lanes, so lane 0 also writes the closing boundary gstart[NG].
    if (lane == 0) gstart[NG] = 64;
    if (lane < NG) {
      int bnd = 0;
      if (lane > 0) {
        const int target = (lane * nnz + NG / 2) / NG;
        int lo = 0, hi = nrows;  // smallest r with estart[r] - e_base >= target
        while (lo < hi) {
          const int mid = (lo + hi) >> 1;
          if (estart[mid] - e_base >= target) hi = mid; else lo = mid + 1;
        }
        bnd = lo;
      }
      gstart[lane] = bnd;
    }
    int lmin = INT_MAX, lmax = -1;  // lane = tile row
    if (fits && lane < nrows)
      for (int k = estart[lane] - e_base; k < estart[lane + 1] - e_base; ++k) {
        lmin = min(lmin, ecol[k]);
        lmax = max(lmax, ecol[k]);
      }
    rmin[lane] = lmin;
    rmax[lane] = lmax;
    if (lane < NG) {  // sender span of each run
      int gmin = INT_MAX, gmax = -1;
      for (int r = gstart[lane]; r < gstart[lane + 1]; ++r) {
        gmin = min(gmin, rmin[r]);
        gmax = max(gmax, rmax[r]);
      }
      gbase[lane] = gmax < 0 ? 0 : gmin;
      if (gmax >= 0 && gmax - gmin >= kDMax) flag[0] = 1;
    }
    if (lane == 0 && !fits) flag[1] = 1;
  }
  __syncthreads();
  int4* dst = reinterpret_cast<int4*>(rec + (long long)t * (kRecBytes / 4));
  dst[tid] = reinterpret_cast<const int4*>(ent)[tid];
}

template <int NTW, bool MULTI>
__global__ __launch_bounds__(512, 1) void transfer_bf16_tiled_kernel(const TransferArgs p) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[kSmemBytes];
  uint16_t* Xs = reinterpret_cast<uint16_t*>(smem);
  float* dt = reinterpret_cast<float*>(smem + kOffDt);
  int* estart = reinterpret_cast<int*>(smem + kOffEnt);
  int* gbase = estart + 65;
  int* ecol = gbase + 64;
  float* ew = reinterpret_cast<float*>(ecol + kEMax);
  int* einfo = reinterpret_cast<int*>(ew + kEMax);
  const int* flag = einfo + kEMax;  // [0] a run too wide for U(0..15), [1] too many entries
  const int* gstart = flag + 4;     // lane group g walks tile rows [gstart[g], gstart[g + 1])
  int* next_item = reinterpret_cast<int*>(smem + kOffNext);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int H = p.H_s;
  // WPH waves share a sender head; each lane group walks a run of rows
  const int WPH = H == 1 ? 8 : H == 2 ? 4 : H <= 4 ? 2 : 1;
  const int n_items = p.tiles_per_lc * p.L_r * 2;
  // The tile's staging record into LDS, one 16-byte-per-lane copy per wave.
  auto copy_record = [&](int item) {
    const Item ni = decode_item(p, item);
    const int* rec = p.tile_rec + (long long)(p.tile_start[ni.b] + ni.tile) * (kRecBytes / 4);
    copy16_to_lds(rec + wave * 256 + 4 * lane, estart + wave * 256);
  };

  // Persistent (interpolating map): the workgroup starts on work item
  // blockIdx.x and takes the next one from the work counter (set to the grid
  // size by the staging kernel) while it builds, so the items in flight stay a
  // contiguous run of the work order, and the next record is copied in during
  // the store.  With concatenated taps (whose per-tap passes leave no registers
  // for the loop) a workgroup does the one item blockIdx.x.
  constexpr bool kPersist = !MULTI;
  int item = blockIdx.x;
  copy_record(item);
  if (p.unrot) {  // U(0..15): rows 0..15 of the sender table, 2 per wave
    const int ri = wave * 2 + (lane >> 5);
    const int c = (lane & 31) ^ (ri & 1);
    copy16_to_lds(p.cs_s + (long long)ri * kDH + 4 * c, dt + wave * 2 * kDH);
  }
  __builtin_amdgcn_s_waitcnt(0);  // both copies have landed
  __syncthreads();

  for (;;) {
  const Item it = decode_item(p, item);
  const Ctx cx = make_ctx(p, it);
  const int Tr = p.Tr[it.b];
  const int j0 = it.tile * 64;
  const int nrows = min(64, Tr - j0);
  const int g0 = p.row0[it.b] + j0;
  const bool unrot = cx.cs_s != nullptr;
  const int e_base = estart[0];
  const bool staged = p.s_extent > 0 && flag[1] == 0 && !(unrot && flag[0] != 0);
  int grabbed = n_items;
  if (kPersist && tid == 0) grabbed = atomicAdd(p.work_ctr, 1);

  f32x16 acc[2][NTW];  // zeroed after the first tap's build
  // This wave's accumulators: receiver head `head`, n-tiles feat[q].
  const int head = NTW == 4 ? wave : (wave >> 1);
  const int nt0 = NTW == 4 ? 0 : (wave & 1);
  constexpr int NTS = 4 / NTW;  // n-tile stride inside the head
  int feat[NTW];
#pragma unroll
  for (int q = 0; q < NTW; ++q) feat[q] = 32 * (nt0 + q * NTS);
  const int KS = H * (kDH / 16);  // k-steps of one tap
  const int NB = p.H_r * (kDH / 32);
  const int lc_store = it.l * 2 + it.c;
  const int ks0 = (int)((unsigned)item % (unsigned)H) * (kDH / 16);  // this item's first k-step

  // One pass per tap of the layer map (MULTI: concatenated taps, each one
  // sender layer): build that tap's X, multiply it by the matching k block of
  // the map into the same accumulators.  From the second tap on the
  // accumulators are live during the build, which then keeps fewer loads in
  // flight.
  const int n_pass = MULTI ? p.n_taps : 1;
  for (int tap = 0; tap < n_pass; ++tap) {
    if (tap > 0) __syncthreads();  // every wave is done reading the previous tap's X
    const Ctx ct = make_ctx(p, it, tap);
    // ---- build X[64][d_in] of this tap ----
    if (staged) {
      const LdsSink xsink{Xs};
      const int sh = wave / WPH;  // sender head this wave builds
      if (sh < H) {
        const GroupLds L{estart, ecol, ew, einfo, dt, e_base};
        const int grp = (wave % WPH) * 8 + (lane >> 3);
        const int r_first = gstart[grp];
        const int rpg = gstart[grp + 1] - r_first;
        const int base = gbase[grp];
        if (MULTI) {  // one sender layer per tap
          if (tap == 0) {
            if (unrot) build_groups<false, true, 3>(ct, p, L, base, sh, r_first, rpg, lane, xsink);
            else build_groups<false, false, 3>(ct, p, L, base, sh, r_first, rpg, lane, xsink);
          } else {
            if (unrot) build_groups<false, true, 2>(ct, p, L, base, sh, r_first, rpg, lane, xsink);
            else build_groups<false, false, 2>(ct, p, L, base, sh, r_first, rpg, lane, xsink);
          }
        } else if (ct.two_tap) {
          if (unrot) build_groups<true, true, 3>(ct, p, L, base, sh, r_first, rpg, lane, xsink);
          else build_groups<true, false, 3>(ct, p, L, base, sh, r_first, rpg, lane, xsink);
        } else {
          if (unrot) build_groups<false, true, 3>(ct, p, L, base, sh, r_first, rpg, lane, xsink);
          else build_groups<false, false, 3>(ct, p, L, base, sh, r_first, rpg, lane, xsink);
        }
      }
    } else {
      const int r = tid >> 3;         // 8 threads per row
      const int e0 = (tid & 7) * 8;   // features e0..e0+7 and e0+64..e0+71 of every head
      for (int h = 0; h < H; ++h) {
        float x[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) x[u] = 0.0f;
        if (r < nrows) build_row_global(p, ct, g0 + r, h, e0, x);
        uint16_t* xr = Xs + r * kXF + h * kDH;
        *reinterpret_cast<uint4*>(xr + e0) = pack8(x);
        *reinterpret_cast<uint4*>(xr + 64 + e0) = pack8(x + 8);
      }
    }
    __syncthreads();
    if (tap == 0) {
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int q = 0; q < NTW; ++q)
#pragma unroll
          for (int i = 0; i < 16; ++i) acc[mt][q][i] = 0.0f;
    }

    // ---- multiply ----
    // The map block of this (layer, role, tap) through a buffer resource: a
    // 32-bit per-lane offset plus the k-step's scalar offset, so a refill costs
    // no 64-bit address arithmetic.
    const bf16x8* Wblk =
        static_cast<const bf16x8*>(p.Wp) + ((long long)lc_store * p.n_taps + tap) * KS * NB * 64;
    const __amdgpu_buffer_rsrc_t rW =
        __builtin_amdgcn_make_buffer_rsrc((void*)Wblk, 0, KS * NB * 64 * 16, 0x00020000);
    const int w_lane = ((4 * head + nt0) * 64 + lane) * 16;  // bytes within a k-step
    bf16x8 wr[4][NTW];  // map fragments of four consecutive k-steps
    auto kstep = [&](int ks) { int k = ks + ks0; return k >= KS ? k - KS : k; };
    auto load_w = [&](bf16x8* dst, int ks) {
      const int k_off = kstep(ks) * NB * 64 * 16;
#pragma unroll
      for (int q = 0; q < NTW; ++q)
        dst[q] = __builtin_bit_cast(
            bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rW, w_lane + q * NTS * 64 * 16, k_off, 0));
    };
    auto read_x = [&](bf16x8* xa, int ks) {
      const int k = kstep(ks);
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
        xa[mt] = *reinterpret_cast<const bf16x8*>(Xs + (32 * mt + (lane & 31)) * kXF + 16 * k +
                                                8 * (lane >> 5));
    };
    bf16x8 xc[2], xn[2];  // X fragments of this k-step and the next
    // One k-step: read next X from LDS, multiply, then refill this map slot with
    // k-step ks + 4.  LOAD is a constant so that the loop body has no branches
    // and every wait on a map fragment keeps the three younger k-steps in flight.
    auto step = [&](bf16x8* wf, int ks, auto load) {
      read_x(xn, ks + 1);
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int q = 0; q < NTW; ++q)
          acc[mt][q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[q], xc[mt], acc[mt][q], 0, 0, 0);
      if (decltype(load)::value) load_w(wf, ks + 4);
      xc[0] = xn[0];
      xc[1] = xn[1];
      __builtin_amdgcn_sched_barrier(0);  // keep the refill in this k-step
    };
    using Load = std::true_type;
    using NoLoad = std::false_type;
#pragma unroll
    for (int u = 0; u < 4; ++u) load_w(wr[u], u);  // KS is a multiple of 8
    read_x(xc, 0);
    for (int ks = 0; ks < KS - 4; ks += 4) {
      step(wr[0], ks, Load());
      step(wr[1], ks + 1, Load());
      step(wr[2], ks + 2, Load());
      step(wr[3], ks + 3, Load());
    }
    step(wr[0], KS - 4, NoLoad());
    step(wr[1], KS - 3, NoLoad());
    step(wr[2], KS - 2, NoLoad());
    step(wr[3], KS - 1, NoLoad());
  }
  if (tid == 0) *next_item = grabbed;
  __syncthreads();  // every wave is done reading X; the X region is free
  const int next = *next_item;

  // ---- store ----
  const bool rot = it.c == 0 && p.rot;
  float* rcs = reinterpret_cast<float*>(smem + kOffRcs);
  float* bias_s = reinterpret_cast<float*>(smem + kOffBias);
  const int d_r = NB * 32;
  if (rot) {  // receiver RoPE rows j0..j0+63: 2 per wave instruction; slot c holds chunk
              // (c & 16) | ((c ^ r) & 15) so that lanes of different rows hit different banks
    for (int q = wave; q < 32; q += 8) {
      const int rr = 2 * q + (lane >> 5);
      const int c = lane & 31;
      const int cs = (c & 16) | ((c ^ rr) & 15);
      const int jr = p.pos0_r[it.b] + j0 + min(rr, nrows - 1);
      copy16_to_lds(p.cs_r + (long long)jr * kDH + 4 * cs, rcs + q * 2 * kDH);
    }
  }
  if (p.bias && wave < d_r / 256)  // 256 floats per wave instruction
    copy16_to_lds(p.bias + (long long)lc_store * d_r + wave * 256 + 4 * lane, bias_s + wave * 256);
  if (next < n_items) copy_record(next);  // this item's record is no longer read
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  uint16_t* stage = reinterpret_cast<uint16_t*>(smem + kOffStage) + wave * 32 * kXS;
  uint16_t* dst_head = static_cast<uint16_t*>(p.R) + it.b * p.r_sb + (long long)it.l * p.r_sl +
                       it.c * p.r_sc + head * p.r_sh;
  float* rsum = reinterpret_cast<float*>(smem + kOffRsum);  // [8 waves][32] row sums of squares
  const float* knorm = (it.c == 0 && p.k_norm) ? p.k_norm + (long long)it.l * kDH : nullptr;
  const int hi4 = 4 * (lane >> 5);
  const int mcol = lane & 31;
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
    const int rl = 32 * mt + mcol;  // tile row held by this lane
    float y[NTW][16];
#pragma unroll
    for (int q = 0; q < NTW; ++q)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float4 bv = make_float4(0.f, 0.f, 0.f, 0.f);
        if (p.bias) bv = *reinterpret_cast<const float4*>(bias_s + head * kDH + feat[q] + 8 * g + hi4);
        y[q][4 * g + 0] = acc[mt][q][4 * g + 0] + bv.x;
        y[q][4 * g + 1] = acc[mt][q][4 * g + 1] + bv.y;
        y[q][4 * g + 2] = acc[mt][q][4 * g + 2] + bv.z;
        y[q][4 * g + 3] = acc[mt][q][4 * g + 3] + bv.w;
      }
    if (knorm) {  // receiver key RMSNorm over each head's 128 features
      float ss = 0.0f;
#pragma unroll
      for (int q = 0; q < NTW; ++q)
#pragma unroll
        for (int i = 0; i < 16; ++i) ss = fmaf(y[q][i], y[q][i], ss);
      ss += __shfl_xor(ss, 32);  // lane ^ 32 holds the same row's other features
      if (NTW == 2) {            // the other half of the head sits in wave ^ 1
        rsum[wave * 32 + mcol] = ss;
        __syncthreads();
        ss += rsum[(wave ^ 1) * 32 + mcol];
        __syncthreads();
      }
      const float inv = 1.0f / sqrtf(ss * (1.0f / kDH) + p.k_norm_eps);
      scale_by_weights<NTW>(y, feat, hi4, knorm, inv);
    }
    if (rot) {
      const float4* crow = reinterpret_cast<const float4*>(rcs) + rl * 32;
#pragma unroll
      for (int q = 0; q < NTW / 2; ++q)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int c = (feat[q] + 8 * g + hi4) >> 2;  // cos chunk, < 16
          const float4 cv = crow[(c ^ rl) & 15];
          const float4 sv = crow[16 | ((c ^ rl) & 15)];
          const float cc[4] = {cv.x, cv.y, cv.z, cv.w};
          const float ss[4] = {sv.x, sv.y, sv.z, sv.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float a = y[q][4 * g + u], b = y[q + NTW / 2][4 * g + u];
            y[q][4 * g + u] = fmaf(a, cc[u], -b * ss[u]);
            y[q + NTW / 2][4 * g + u] = fmaf(b, cc[u], a * ss[u]);
          }
        }
    }
#pragma unroll
    for (int q = 0; q < NTW; ++q)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint2 v = make_uint2(pack2(y[q][4 * g], y[q][4 * g + 1]), pack2(y[q][4 * g + 2], y[q][4 * g + 3]));
        *reinterpret_cast<uint2*>(stage + mcol * kXS + 32 * q + 8 * g + hi4) = v;
      }
    constexpr int LPR = NTW * 4;  // lanes per row, 16 bytes each
    constexpr int RPP = 64 / LPR;
#pragma unroll
    for (int pass = 0; pass < 32 / RPP; ++pass) {
      const int rr = pass * RPP + lane / LPR;
      const int ci = lane % LPR;
      const uint4 v = *reinterpret_cast<const uint4*>(stage + rr * kXS + 8 * ci);
      const int jj = j0 + 32 * mt + rr;
      if (jj < Tr)  // streaming store: the receiver rows are not read again here, so
                    // they should not push the shared map out of L2
        __builtin_nontemporal_store(
            u32x4{v.x, v.y, v.z, v.w},
            reinterpret_cast<u32x4*>(dst_head + (long long)jj * p.r_st + feat[ci / 4] + 8 * (ci % 4)));
    }
  }
  if (!kPersist || next >= n_items) break;
  __syncthreads();  // every wave is done with the staging rows; the next build writes X
  item = next;
  }
}

// ---------------------------------------------------------------------------
// Staged path, build: the aligned features of one (slab, 64-row tile) written
// to global memory in the layout the staged GEMM reads.  The tile is built in
// LDS and then written out: in the slab's [256-row tile][k-tile][256][32]
// layout its rows are one 4 KB run per k-tile, so every wave store is 1 KB of
// whole lines (rows past the sequence end carry zeros the GEMM never stores).
// Each wave writes its own sender head as soon as its walk ends.  A slab is (role,
// receiver layer) for the interpolating map -- x_j of Sec. 3.1 with the layer
// weights of its two taps -- or (role, sender layer) for concatenated taps --
// one block x_j^t of Eq. 2, shared by every receiver layer that reads that
// sender layer.  The arithmetic is the fused kernel's build (same staging
// record, same group walk, one bf16 rounding per feature).
// ---------------------------------------------------------------------------
// 16 bytes from LDS to global memory as a streaming (non-temporal) store: the
// slab is read back only after the whole build, so it need not stay in L2.
__device__ __forceinline__ void nt_store16(uint16_t* g, const uint16_t* l) {
  typedef unsigned v4u __attribute__((ext_vector_type(4)));
  __builtin_nontemporal_store(*reinterpret_cast<const v4u*>(l), reinterpret_cast<v4u*>(g));
}

__global__ __launch_bounds__(512) void staged_build_kernel(const TransferArgs p) {
  __shared__ __attribute__((aligned(16))) uint16_t xl[64 * kXF];  // the built tile, fused-kernel layout
  __shared__ __attribute__((aligned(16))) int ent[kRecBytes / 4];
  __shared__ __attribute__((aligned(16))) float dt[kDMax * kDH];
  int* estart = ent;
  int* gbase = estart + 65;
  int* ecol = gbase + 64;
  float* ew = reinterpret_cast<float*>(ecol + kEMax);
  int* einfo = reinterpret_cast<int*>(ew + kEMax);
  const int* flag = einfo + kEMax;
  const int* gstart = flag + 4;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  const int slab = blockIdx.x / p.tiles_per_lc;  // (role, layer), role-major
  const int t = blockIdx.x - slab * p.tiles_per_lc;
  Item it;
  it.c = slab / p.n_slab_layers;
  it.l = slab - it.c * p.n_slab_layers;
  int b = 0;
  while (b + 1 < p.B && p.tile_start[b + 1] <= t) ++b;
  it.b = b;
  it.tile = t - p.tile_start[b];
  Ctx cx;
  if (p.concat) {  // one sender layer, weight 1
    const uint16_t* Sb = static_cast<const uint16_t*>(p.S) + it.b * p.s_sb + it.c * p.s_sc;
    cx.S_lo = cx.S_hi = Sb + (long long)it.l * p.s_sl;
    cx.cs_s = (it.c == 0 && p.unrot) ? p.cs_s + (long long)p.pos0_s[it.b] * kDH : nullptr;
    cx.wlo = 1.0f;
    cx.whi = 0.0f;
    cx.two_tap = false;
    cx.Ts = p.Ts[it.b];
  } else {
    cx = make_ctx(p, it);
  }
  // Keys un-rotate at the sender positions when the call asks for it; values
  // never do (their context carries no sender table).
  const bool unrot = cx.cs_s != nullptr;
  copy16_to_lds(p.tile_rec + (long long)t * (kRecBytes / 4) + wave * 256 + 4 * lane, estart + wave * 256);
  if (unrot) {  // U(0..15): rows 0..15 of the sender table, 2 per wave
    const int ri = wave * 2 + (lane >> 5);
    const int c = (lane & 31) ^ (ri & 1);
    copy16_to_lds(p.cs_s + (long long)ri * kDH + 4 * c, dt + wave * 2 * kDH);
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  const int Tr = p.Tr[it.b];
  const int j0 = it.tile * 64;
  const int nrows = min(64, Tr - j0);
  const int g0 = p.row0[it.b] + j0;
  const LdsSink sink{xl};
  const int rt = p.rt_start[it.b] + (it.tile >> 2);
  uint16_t* dst = p.xs + slab * p.xs_slab + (long long)rt * (kStagedRows * kHMax * kDH) +
                  (it.tile & 3) * 64 * 32;
  const bool staged = p.s_extent > 0 && flag[1] == 0 && !(unrot && flag[0] != 0);
  if (staged) {  // eight sender heads: wave w builds head w
    const GroupLds L{estart, ecol, ew, einfo, dt, estart[0]};
    const int grp = lane >> 3;
    const int r_first = gstart[grp], rpg = gstart[grp + 1] - r_first, base = gbase[grp];
    if (cx.two_tap && unrot) build_groups<true, true, 3>(cx, p, L, base, wave, r_first, rpg, lane, sink);
    else if (cx.two_tap) build_groups<true, false, 3>(cx, p, L, base, wave, r_first, rpg, lane, sink);
    else if (unrot) build_groups<false, true, 3>(cx, p, L, base, wave, r_first, rpg, lane, sink);
    else build_groups<false, false, 3>(cx, p, L, base, wave, r_first, rpg, lane, sink);
    // The wave's own head (k-tiles 4 wave .. 4 wave + 3 of the 64 rows) goes
    // out as soon as its walk ends: LDS operations of one wave run in order.
    const int c8 = (lane & 3) * 8;
#pragma unroll 4
    for (int i = 0; i < 16; ++i) {
      const int kt = 4 * wave + (i >> 2), r = 16 * (i & 3) + (lane >> 2);
      nt_store16(dst + kt * (kStagedRows * 32) + r * 32 + c8, xl + r * kXF + kt * 32 + c8);
    }
  } else {
    const int r = tid >> 3;        // 8 threads per row
    const int e0 = (tid & 7) * 8;  // features e0..e0+7 and e0+64..e0+71 of every head
    for (int h = 0; h < kHMax; ++h) {
      float x[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) x[u] = 0.0f;
      if (r < nrows) build_row_global(p, cx, g0 + r, h, e0, x);
      sink(r, h * kDH + e0, pack8(x));
      sink(r, h * kDH + 64 + e0, pack8(x + 8));
    }
    __syncthreads();
    const int r2 = (tid & 255) >> 2, c8 = (tid & 3) * 8;
#pragma unroll 4
    for (int kt = tid >> 8; kt < kHMax * kDH / 32; kt += 2)
      nt_store16(dst + kt * (kStagedRows * 32) + r2 * 32 + c8, xl + r2 * kXF + kt * 32 + c8);
  }
}

// ---------------------------------------------------------------------------
// bf16 transfer kernel, direct (d_h = 128, WN receiver heads): the same
// computation with X built straight from global memory and one workgroup per
// 64 (8/WN) rows.  Used for two receiver heads, where a 64-row tile over 8
// waves would split a RoPE pair across lanes.
// ---------------------------------------------------------------------------
template <int WN>
__global__ __launch_bounds__(512, 1) void transfer_bf16_direct_kernel(const TransferArgs p) {
  constexpr int WM = 8 / WN;
  constexpr int MT = 64 * WM;
  constexpr int XBUF = MT * kXS;
  constexpr int STAGE = 32 * kXS;
  constexpr int LDS = (2 * XBUF > 8 * STAGE) ? 2 * XBUF : 8 * STAGE;
  __shared__ __attribute__((aligned(16))) uint16_t lds[LDS];

  const Item it = decode_item(p, blockIdx.x);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int j0 = it.tile * MT;
  const int Tr = p.Tr[it.b];
  const int row0 = p.row0[it.b];
  const int KS = p.n_taps * p.H_s * (kDH / 16);  // k-steps of the whole map row
  const int NB = p.H_r * (kDH / 32);
  const int lc_store = it.l * 2 + it.c;
  // Map fragments through a buffer resource over this (layer, role)'s block.
  const __amdgpu_buffer_rsrc_t rW = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(static_cast<const bf16x8*>(p.Wp) + (long long)lc_store * KS * NB * 64), 0,
      KS * NB * 64 * 16, 0x00020000);
  const int w_lane = ((wn * 4) * 64 + lane) * 16;  // bytes
  const int brow = tid >> 3;
  const int e0 = (tid & 7) * 8;

  f32x16 acc[2][4];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[mt][nt][i] = 0.0f;

  // v runs over (tap, sender head) pairs: the k blocks of the map row
  for (int v = 0; v < p.n_taps * p.H_s; ++v) {
    const int h = v % p.H_s;
    const Ctx cx = make_ctx(p, it, v / p.H_s);
    uint16_t* xb = lds + (v & 1) * XBUF;
#pragma unroll
    for (int q = 0; q < WM; ++q) {
      const int r = brow + 64 * q;
      float x[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) x[u] = 0.0f;
      if (j0 + r < Tr) build_row_global(p, cx, row0 + j0 + r, h, e0, x);
      *reinterpret_cast<uint4*>(xb + r * kXS + e0) = pack8(x);
      *reinterpret_cast<uint4*>(xb + r * kXS + e0 + 64) = pack8(x + 8);
    }
    __syncthreads();
    const int v_off = v * 8 * NB * 64 * 16;  // k-steps of block v
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      bf16x8 xa[2], wf[4];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
        xa[mt] = *reinterpret_cast<const bf16x8*>(
            xb + (64 * wm + 32 * mt + (lane & 31)) * kXS + 16 * s + 8 * (lane >> 5));
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
        wf[nt] = __builtin_bit_cast(
            bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rW, w_lane + (s * NB + nt) * 64 * 16, v_off, 0));
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[nt], xa[mt], acc[mt][nt], 0, 0, 0);
    }
  }
  __syncthreads();  // every wave is done reading X; LDS becomes staging space

  const int feat[4] = {0, 32, 64, 96};
  uint16_t* stage = lds + wave * STAGE;
  uint16_t* dst_head = static_cast<uint16_t*>(p.R) + it.b * p.r_sb + (long long)it.l * p.r_sl +
                       it.c * p.r_sc + wn * p.r_sh;
  const float* bias_head = p.bias ? p.bias + (long long)lc_store * NB * 32 + wn * kDH : nullptr;
  const bool rot = it.c == 0 && p.rot;
  const float* cr = rot ? p.cs_r + (long long)p.pos0_r[it.b] * kDH : nullptr;
  const float* knorm = (it.c == 0 && p.k_norm) ? p.k_norm + (long long)it.l * kDH : nullptr;
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
    epilogue_rows<4>(p, acc[mt], feat, bias_head, cr, rot, knorm, stage, dst_head,
                     j0 + 64 * wm + 32 * mt, Tr, lane);
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
  const int NV = p.n_taps * p.H_s;  // (tap, sender head) blocks of the map row
  const int d_in = NV * d, d_r = p.H_r * d;
  const int j0 = it.tile * RT;
  const int Tr = p.Tr[it.b], Ts = p.Ts[it.b];
  const bool keys = it.c == 0;
  const bool unrot = keys && p.unrot, rot = keys && p.rot;
  const float sr = p.inv_r ? p.inv_r[it.l * 2 + it.c] : 1.0f;  // the map sees x / r
  const float wlo = p.wlo[it.l] * sr, whi = p.whi[it.l] * sr;
  const bool two_tap = p.whi[it.l] != 0.0f;
  const float* Sb = static_cast<const float*>(p.S) + it.b * p.s_sb + it.c * p.s_sc;
  const int lc_store = it.l * 2 + it.c;

  for (int idx = threadIdx.x; idx < RT * NV * half; idx += kF32Threads) {
    const int r = idx / (NV * half);
    const int rem = idx - r * (NV * half);
    const int vh = rem / half, f = rem - vh * half;
    const int h = vh % p.H_s, t = vh / p.H_s;
    const int lo = p.concat ? p.taps[it.l][t] : p.lo[it.l];
    const float* S_lo = Sb + (long long)lo * p.s_sl;
    const float* S_hi = Sb + (long long)(p.concat ? lo : p.hi[it.l]) * p.s_sl;
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
          const float* cs = p.cs_s + (long long)(p.pos0_s[it.b] + i) * d;
          const float c = cs[f], s = cs[half + f];
          const float u1 = fmaf(m1, c, m2 * s);
          const float u2 = fmaf(m2, c, -m1 * s);
          m1 = u1;
          m2 = u2;
        }
        x1 = fmaf(w, m1, x1);
        x2 = fmaf(w, m2, x2);
      }
    }
    xs[r * d_in + vh * d + f] = x1;
    xs[r * d_in + vh * d + f + half] = x2;
  }
  __syncthreads();

  const float* W = static_cast<const float*>(p.Wp) + (long long)lc_store * d_r * d_in;
  float* Rb = static_cast<float*>(p.R) + it.b * p.r_sb + (long long)it.l * p.r_sl + it.c * p.r_sc;
  constexpr int kMaxRT = 16;
  const float* knorm = (keys && p.k_norm) ? p.k_norm + (long long)it.l * d : nullptr;
  // Every thread takes the same number of trips (pc past the end computes
  // nothing and stores nothing), so the key norm's shuffles see whole waves;
  // the half = d/2 threads of one receiver head are consecutive lanes.
  for (int pc0 = 0; pc0 < p.H_r * half; pc0 += kF32Threads) {
    const int pc = pc0 + threadIdx.x;
    const bool live = pc < p.H_r * half;
    const int hr = live ? pc / half : 0, f = live ? pc - hr * half : 0;
    const int n1 = hr * d + f, n2 = n1 + half;
    float y1[kMaxRT], y2[kMaxRT];
#pragma unroll
    for (int r = 0; r < kMaxRT; ++r) y1[r] = y2[r] = 0.f;
    const float* W1 = W + (long long)n1 * d_in;
    const float* W2 = W + (long long)n2 * d_in;
    for (int k = 0; k < (live ? d_in : 0); ++k) {
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
    const float b1 = (p.bias && live) ? p.bias[(long long)lc_store * d_r + n1] : 0.f;
    const float b2 = (p.bias && live) ? p.bias[(long long)lc_store * d_r + n2] : 0.f;
    const float g1 = knorm ? knorm[f] : 1.f, g2 = knorm ? knorm[f + half] : 1.f;
#pragma unroll
    for (int r = 0; r < kMaxRT; ++r) {
      const int j = j0 + r;
      if (r >= RT) continue;  // uniform: the shuffles below stay whole-wave
      float v1 = y1[r] + b1, v2 = y2[r] + b2;
      if (knorm) {  // RMSNorm over the head's d features, held by half lanes
        float ss = fmaf(v1, v1, v2 * v2);
        for (int o = 1; o < half; o <<= 1) ss += __shfl_xor(ss, o);
        const float inv = 1.0f / sqrtf(ss / (float)d + p.k_norm_eps);
        v1 *= inv * g1;
        v2 *= inv * g2;
      }
      if (!live || j >= Tr) continue;
      if (rot) {
        const float* cs = p.cs_r + (long long)(p.pos0_r[it.b] + j) * d;
        const float c = cs[f], s = cs[half + f];
        const float u1 = fmaf(v1, c, -v2 * s);
        const float u2 = fmaf(v2, c, v1 * s);
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

int transfer_rows_per_tile(int dtype, int H_r, int H_s, int n_taps, int d_h) {
  if (dtype == HF_BF16)
    return ((H_r == 4 || H_r == 8) && H_s <= kHMax) ? 64 : 64 * (8 / (H_r > 0 ? H_r : 1));
  const int d_in = n_taps * H_s * d_h;
  int rt = 8192 / (d_in > 0 ? d_in : 1);  // fp32 X tile <= 32 KB of LDS
  return rt < 1 ? 1 : (rt > 16 ? 16 : rt);
}

static bool uses_tiled(int dtype, int H_r, int H_s, int d_h) {
  return dtype == HF_BF16 && d_h == kDH && (H_r == 4 || H_r == 8) && H_s <= kHMax;
}

size_t transfer_tile_record_bytes(int dtype, int H_r, int H_s, int d_h) {
  return uses_tiled(dtype, H_r, H_s, d_h) ? kRecBytes : 0;
}

int transfer_persistent_grid(const TransferArgs& a, int n_cu) {
  const long long items = (long long)a.tiles_per_lc * a.L_r * 2;
  return (int)(items < n_cu ? items : n_cu);
}

hipError_t launch_transfer_stage(int dtype, const TransferArgs& a, hipStream_t s) {
  const int tiles = a.tile_start[a.B];
  if (!uses_tiled(dtype, a.H_r, a.H_s, a.d_h) || tiles <= 0) return hipSuccess;
  if (!a.tile_rec) return hipErrorInvalidValue;
  if (!a.work_ctr || a.n_wg < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(stage_tiles_kernel, dim3((unsigned)tiles), dim3(512), 0, s, a,
                     const_cast<int*>(a.tile_rec));
  return hipGetLastError();
}

hipError_t launch_rope_table(float* tab, int P, int d_h, double theta, hipStream_t s) {
  const int half = d_h / 2;
  const long long n = (long long)P * half;
  if (n <= 0) return hipSuccess;
  const dim3 grid((unsigned)((P + 4 * kRopePpt - 1) / (4 * kRopePpt)), (unsigned)((half + 63) / 64));
  hipLaunchKernelGGL(rope_table_kernel, grid, dim3(64, 4), 0, s, tab, P, half, d_h, theta);
  return hipGetLastError();
}

hipError_t launch_pack_maps(int dtype, int n_lc, int d_r, int d_in, const void* A, void* A_packed,
                            hipStream_t s) {
  static_assert(HF_PACKED_HEADER_BYTES == 64 * 4, "header kernel writes 64 words");
  hipLaunchKernelGGL(pack_header_kernel, dim3(1), dim3(64), 0, s, static_cast<uint32_t*>(A_packed),
                     dtype, n_lc / 2, d_r, d_in);
  void* Wp = static_cast<char*>(A_packed) + HF_PACKED_HEADER_BYTES;
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

// ---------------------------------------------------------------------------
// Scratch of hf_transfer_kv_noalloc: the workspace of a transfer (RoPE
// tables, staged tile records, work counter) in a file-scope device array, so
// that the call allocates nothing.  Each device holds its own copy from module
// load until the process ends.  Host code never passes the array's name to a
// kernel: it resolves the device address once per device and uses that.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[HF_NOALLOC_SCRATCH_BYTES];

hipError_t noalloc_scratch(void** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* per_device[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(mu);
  if (!per_device[dev]) {  // first call on this device, with it current
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    per_device[dev] = p;
  }
  *ptr = per_device[dev];
  return hipSuccess;
}

bool staged_supported(int dtype, int H_s, int H_r, int d_h) {
  return dtype == HF_BF16 && d_h == kDH && H_s == kHMax && H_r == kHMax;
}

hipError_t launch_staged_build(const TransferArgs& a, hipStream_t s) {
  const long long items = (long long)a.tiles_per_lc * a.n_slab_layers * 2;
  if (items <= 0) return hipSuccess;
  if (!a.xs || !a.tile_rec || items > INT32_MAX) return hipErrorInvalidValue;
  const dim3 grid((unsigned)items);
  hipLaunchKernelGGL(staged_build_kernel, grid, dim3(512), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_transfer(int dtype, const TransferArgs& a, hipStream_t s) {
  const long long items = (long long)a.tiles_per_lc * a.L_r * 2;
  if (items <= 0) return hipSuccess;
  const dim3 grid((unsigned)items);
  const bool tiled = uses_tiled(dtype, a.H_r, a.H_s, a.d_h);
  if (tiled && (!a.tile_rec || !a.work_ctr || a.n_wg < 1)) return hipErrorInvalidValue;
  const dim3 pgrid((unsigned)a.n_wg);  // persistent (interpolating map): one workgroup per CU
  if (dtype == HF_BF16) {
    switch (a.H_r) {
      case 2: hipLaunchKernelGGL(transfer_bf16_direct_kernel<2>, grid, dim3(512), 0, s, a); break;
      case 4:
        if (tiled && a.concat)
          hipLaunchKernelGGL((transfer_bf16_tiled_kernel<2, true>), grid, dim3(512), 0, s, a);
        else if (tiled)
          hipLaunchKernelGGL((transfer_bf16_tiled_kernel<2, false>), pgrid, dim3(512), 0, s, a);
        else hipLaunchKernelGGL(transfer_bf16_direct_kernel<4>, grid, dim3(512), 0, s, a);
        break;
      case 8:
        if (tiled && a.concat)
          hipLaunchKernelGGL((transfer_bf16_tiled_kernel<4, true>), grid, dim3(512), 0, s, a);
        else if (tiled)
          hipLaunchKernelGGL((transfer_bf16_tiled_kernel<4, false>), pgrid, dim3(512), 0, s, a);
        else hipLaunchKernelGGL(transfer_bf16_direct_kernel<8>, grid, dim3(512), 0, s, a);
        break;
      default: return hipErrorInvalidValue;
    }
  } else {
    const size_t shmem = (size_t)a.rows_per_tile * a.n_taps * a.H_s * a.d_h * sizeof(float);
    hipLaunchKernelGGL(transfer_f32_kernel, grid, dim3(kF32Threads), shmem, s, a);
  }
  return hipGetLastError();
}

}  // namespace hf
