// Staged transfer path, multiply: y_j = A[l, c] x_j + b[l, c] over all
// (layer, role) pairs (Eq. 9), from the aligned features the staged build wrote,
// with the receiver RoPE in the epilogue and the result written straight into
// the receiver cache layout [L_R, 2, H_kv, T, d_h].
//
// A persistent bf16 GEMM for gfx950.  One workgroup per CU, 8 waves (2 per
// SIMD), a 256-row x 256-feature output tile per work item: wave w owns rows
// 64 (w >> 1) .. +64 and receiver head 2 nt + (w & 1), 128 fp32 accumulators
// per lane on v_mfma_f32_32x32x16_bf16 (the map fragment is operand A, the
// feature fragment operand B, so a lane holds four consecutive output features
// of one row and a RoPE pair (f, f + 64) sits in one lane).  The k-loop streams
// 32-feature k-tiles of both operands into four LDS stages with direct
// buffer->LDS loads issued three k-tiles ahead; the feature slab is stored
// k-tile-major by the build, so every stage fill is whole 16 KB blocks.  Work
// items are dealt out so that the four feature tiles of one row tile run on
// one XCD (workgroup i runs on XCD i % 8), where they share the row tile in L2.
#include <hip/hip_runtime.h>

#include <cstddef>

#include "hf_internal.h"

namespace hf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;

#define FI __device__ __forceinline__
#define SB() __builtin_amdgcn_sched_barrier(0)

constexpr int kBM = kStagedRows;  // rows per tile
constexpr int kBK = 32;           // features per k-tile
constexpr int kWSt = 16384;       // map part of a stage: 2 k-steps x 8 fragments x 1 KB
constexpr int kSlabTile = kBM * 1024;  // elements of one 256-row tile of a slab (1024 features)
constexpr int kMB = 2;            // 32-row blocks per wave

// s_waitcnt immediate that waits until at most n vector-memory operations are
// outstanding and leaves the other counters alone (gfx9 encoding).
constexpr int wait_vm(int n) { return (n & 0xF) | ((n >> 4) << 14) | (7 << 4) | (0xF << 8); }

FI uint32_t pack2(float a, float b) {
  bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// A buffer resource from a pointer every lane holds, built in scalar registers.
FI __amdgpu_buffer_rsrc_t mk_rsrc(const void* p, int bytes) {
  const uint64_t v = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return __builtin_amdgcn_make_buffer_rsrc((void*)(((uint64_t)hi << 32) | lo), 0,
                                           __builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}

// An opaque copy: values derived from it are formed where it is, not hoisted.
FI int opaque(int x) {
  asm volatile("" : "+v"(x));
  return x;
}

// Feature rows inside a stage: row r of a k-tile is 64 bytes, its 16-byte chunk
// c stored at slot c ^ sw(r), so that the 32 rows one fragment read touches
// fall on distinct banks.
FI int sw(int r) { return ((r >> 1) ^ (r >> 3)) & 3; }

struct Lane {
  int wave, lane, wr, wc, hi4;
  int vw;        // map DMA: this lane's 16 bytes of a fragment
  int vt0, vt1;  // feature DMA: this lane's row and chunk in a 16-row block (block parity 0 / 1)
  int xo0, xo1;  // feature fragment offsets in a stage (k-step 0 / 1)
  int wo;        // map fragment offset in a stage
};

// One work item: a 256-row x 256-feature output tile of one (layer, role).
struct Job {
  const uint16_t* wb;     // packed maps of the (layer, role), fragment order
  const uint16_t* xt0;    // the 256-row feature tile of each tap (1024 features, k-tile-major)
  const uint16_t* xt1;
  const uint16_t* xt2;
  const float* bias;      // the tile's 256 bias values, or nullptr
  uint16_t* rbase;        // receiver cache at (sequence, layer, role, head 2 nt, row 0)
  int nt, j0, Tr, pos0, keys, l;
};

// Byte i of a kernel-argument byte array, read as the aligned dword that holds
// it: gfx950 has no scalar byte loads, and a vector load here would wait (in
// order) for every load and store in flight.
static_assert(offsetof(TransferArgs, taps) % 4 == 0, "taps must be dword aligned");
FI int arg_byte(const uint8_t* base, int i) {
  i = __builtin_amdgcn_readfirstlane(i);
  const uint32_t w = reinterpret_cast<const uint32_t*>(base)[i >> 2];
  return (int)((w >> (8 * (i & 3))) & 0xffu);
}

FI Job decode(const TransferArgs& p, int xcd, int jj) {
  Job J;
  const int q = 8 * (jj >> 2) + xcd;  // (layer-role, row tile) quad, role-major
  const int lc = q / p.n_rt;
  const int rt = q - lc * p.n_rt;
  const int c = lc / p.L_r;
  const int l = lc - c * p.L_r;
  const int lm = l * 2 + c;  // the (layer, role) index of the packed maps and the bias
  J.nt = jj & 3;
  int b = 0;
  while (b + 1 < p.B && p.rt_start[b + 1] <= rt) ++b;
  J.j0 = (rt - p.rt_start[b]) * kBM;
  J.Tr = p.Tr[b];
  J.pos0 = p.pos0_r[b];
  J.keys = c == 0;
  J.wb = static_cast<const uint16_t*>(p.Wp) + (long long)lm * (p.n_taps * 64) * 32 * 512;
  const uint16_t* xrt = p.xs + (long long)c * p.n_slab_layers * p.xs_slab + (long long)rt * kSlabTile;
  const int t1 = p.n_taps > 1 ? 1 : 0, t2 = p.n_taps > 2 ? 2 : 0;
  const uint8_t* tp = &p.taps[0][0];
  J.xt0 = xrt + (long long)(p.concat ? arg_byte(tp, 3 * l) : l) * p.xs_slab;
  J.xt1 = xrt + (long long)(p.concat ? arg_byte(tp, 3 * l + t1) : l) * p.xs_slab;
  J.xt2 = xrt + (long long)(p.concat ? arg_byte(tp, 3 * l + t2) : l) * p.xs_slab;
  J.bias = p.bias ? p.bias + (long long)lm * 1024 + J.nt * 256 : nullptr;
  J.l = l;
  J.rbase = static_cast<uint16_t*>(p.R) + b * p.r_sb + (long long)l * p.r_sl + c * p.r_sc +
            (long long)(2 * J.nt) * p.r_sh;
  return J;
}

// Stage fills for k-tile kt (2 map fragments and 2 16-row feature blocks per
// wave, straight into LDS).
FI void dma_w(const Lane& L, const uint16_t* wb, int wbytes, int nt, int kt, unsigned char* sb, int i) {
  const __amdgpu_buffer_rsrc_t rW = mk_rsrc(wb, wbytes);
  const int f = 2 * L.wave + i;  // 0..15: k-step f >> 3, fragment f & 7
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rW, (lds_void_t*)(sb + f * 1024), 16, L.vw,
                                           ((2 * kt + (f >> 3)) * 32 + 8 * nt + (f & 7)) * 1024, 0, 0);
}
FI void dma_x(const Lane& L, const uint16_t* xt, int kt, unsigned char* sb, int i) {
  const __amdgpu_buffer_rsrc_t rX = mk_rsrc(xt, kSlabTile * 2);
  const int blk = 2 * L.wave + i;  // 16-row block 0..15
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rX, (lds_void_t*)(sb + kWSt + blk * 1024), 16,
                                           (i & 1) ? L.vt1 : L.vt0, (kt & 31) * kBM * kBK * 2 + i * 1024,
                                           0, 0);
}
// The tap of k-tile kt.  The three pointers pass through an opaque copy before
// the select: a select between two fields of J would otherwise become one
// load at a computed field address, which keeps the whole work item in
// scratch memory and stores it there once per item.
FI const uint16_t* opaque_ptr(const uint16_t* q) {
  asm volatile("" : "+v"(q));
  return q;
}
FI const uint16_t* tap_tile(const Job& J, int kt) {
  const int t = kt >> 5;
  const uint16_t* a = opaque_ptr(J.xt0);
  const uint16_t* b = opaque_ptr(J.xt1);
  const uint16_t* c = opaque_ptr(J.xt2);
  return t == 0 ? a : t == 1 ? b : c;
}
FI void dma_all(const Lane& L, const Job& J, int wbytes, int kt, unsigned char* sb) {
  dma_w(L, J.wb, wbytes, J.nt, kt, sb, 0);
  dma_w(L, J.wb, wbytes, J.nt, kt, sb, 1);
  dma_x(L, tap_tile(J, kt), kt, sb, 0);
  dma_x(L, tap_tile(J, kt), kt, sb, 1);
}

FI void rd_frags(const Lane& L, const unsigned char* sb, int ks, bf16x8 (&fx)[kMB], bf16x8 (&fw)[4]) {
  const int xo = ks ? L.xo1 : L.xo0;
#pragma unroll
  for (int m = 0; m < kMB; ++m) fx[m] = *reinterpret_cast<const bf16x8*>(sb + xo + m * 2048);
#pragma unroll
  for (int q = 0; q < 4; ++q) fw[q] = *reinterpret_cast<const bf16x8*>(sb + ks * 8192 + L.wo + q * 1024);
}
// ZERO: the first k-step of a work item, which starts the accumulators from 0.
template <bool ZERO>
FI void mfma4(f32x16 (&acc)[kMB][4], const bf16x8 (&fx)[kMB], const bf16x8 (&fw)[4], int m) {
  const f32x16 zero = {};
#pragma unroll
  for (int q = 0; q < 4; ++q)
    acc[m][q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[q], fx[m], ZERO ? zero : acc[m][q], 0, 0, 0);
}

// One k-tile.  f0x/f0w hold its k-step-0 fragments (read during the previous
// k-tile); sb is its stage, sn the next k-tile's, sd the stage that k-tile kd
// of job D (this job's k-tile kt + 3, or the next job's first ones) is loaded
// into.  The wait lets at most NV vector-memory operations of this wave stay
// outstanding, so that its loads of k-tile kt + 1 have landed: in steady state
// only the 4 loads of k-tile kt + 2 were issued after them; in the first two
// k-tiles of a work item the previous item's 16 receiver-row stores (and the
// bias and RoPE-row loads of waves 0..3) were issued after them too.  FIRST:
// k-tile 0 of a work item.  The issue order is fixed: fragments for k-step 1,
// then each group of 4 MFMAs after one stage load.
template <int NV, bool FIRST>
FI void ktile(const Lane& L, f32x16 (&acc)[kMB][4], bf16x8 (&f0x)[kMB], bf16x8 (&f0w)[4], bool more,
              unsigned char* sb, unsigned char* sn, unsigned char* sd, const Job& D, int wbytes, int kd) {
  __builtin_amdgcn_s_waitcnt(wait_vm(NV));
  __builtin_amdgcn_s_barrier();  // ... for every wave; stage sd is no longer read
  SB();
  bf16x8 f1x[kMB], f1w[4];
  rd_frags(L, sb, 1, f1x, f1w);
  SB();
  const uint16_t* xt = tap_tile(D, kd);
#pragma unroll
  for (int m = 0; m < kMB; ++m) {
    dma_w(L, D.wb, wbytes, D.nt, kd, sd, m);
    mfma4<FIRST>(acc, f0x, f0w, m);
    SB();
  }
  if (more) rd_frags(L, sn, 0, f0x, f0w);
  SB();
#pragma unroll
  for (int m = 0; m < kMB; ++m) {
    dma_x(L, xt, kd, sd, m);
    mfma4<false>(acc, f1x, f1w, m);
    SB();
  }
}

// Staging accesses of the epilogue, written as instructions the compiler does
// not see as LDS accesses.  Stage 3 was last filled by a load into LDS that the
// explicit waits have completed, but the compiler cannot tell which load in
// flight targets which stage and would wait for all of them, the next work
// item's k-tiles included.  The four reads end with their own wait.
FI uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}
FI void stg_write8(uint32_t a, uint2 v) {
  asm volatile("ds_write_b64 %0, %1" : : "v"(a), "v"(v) : "memory");
}
FI void stg_read4x16(const uint32_t (&a)[4], u32x4 (&v)[4]) {
  asm volatile(
      "ds_read_b128 %0, %4\n\t"
      "ds_read_b128 %1, %5\n\t"
      "ds_read_b128 %2, %6\n\t"
      "ds_read_b128 %3, %7\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3])
      : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3])
      : "memory");
}

// RoPE angles of the lane's row as a sum: the row's 32-row block base (st0 row)
// plus its offset r < 32 in the block (st1 row r, stored with chunk c of row r
// at slot c ^ r).  cos(a + b) = cos a cos b - sin a sin b and
// sin(a + b) = sin a cos b + cos a sin b, in fp32 (about 3 ulp of error).
FI void rope_cs(const Lane& L, const float* st0row, const float* st1, int qq, int g, f32x4& c,
                f32x4& sn) {
  const int r = L.lane & 31;
  const int k = 32 * qq + 8 * g + L.hi4;
  const f32x4 c0 = *reinterpret_cast<const f32x4*>(st0row + k);
  const f32x4 s0 = *reinterpret_cast<const f32x4*>(st0row + 64 + k);
  const f32x4 c1 = *reinterpret_cast<const f32x4*>(st1 + r * 128 + (((k >> 2) ^ r) << 2));
  const f32x4 s1 = *reinterpret_cast<const f32x4*>(st1 + r * 128 + ((((k >> 2) + 16) ^ r) << 2));
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    c[u] = fmaf(c0[u], c1[u], -s0[u] * s1[u]);
    sn[u] = fmaf(s0[u], c1[u], c0[u] * s1[u]);
  }
}

// One 32-row block of the wave's 64 x 128 tile: bias, receiver RoPE (ROT),
// bf16, then two staged passes that each write 64 features of the 32 rows as
// 128-byte row halves.  Staging row rr keeps its 16-byte chunk c at slot
// c ^ ((rr >> 1) & 7): the 32 rows of one 8-byte write then cover 16 distinct
// 16-byte bank groups, the most a 128-byte row stride allows.
template <bool ROT, bool KN, int m>
FI void epi_block(const Lane& L, const f32x16 (&acc)[kMB][4], int j0, int Tr, long long r_st,
                  const float* bsh, float scale, const float* knh, float eps, uint16_t* stg,
                  __amdgpu_buffer_rsrc_t rR, const float* st0, const float* st1) {
  const int rr = L.lane & 31;
  float keep[2][4][4];
  uint2 v0[2][4];
  float inv = 1.0f;
  if (KN) {  // receiver key RMSNorm over the head's 128 features (lanes l and l ^ 32)
    float ss = 0.0f;
#pragma unroll
    for (int qq = 0; qq < 2; ++qq)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 b0 = *reinterpret_cast<const f32x4*>(bsh + 32 * qq + 8 * g);
        const f32x4 b1 = *reinterpret_cast<const f32x4*>(bsh + 64 + 32 * qq + 8 * g);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float y0 = fmaf(acc[m][qq][4 * g + u], scale, b0[u]);
          const float y1 = fmaf(acc[m][qq + 2][4 * g + u], scale, b1[u]);
          ss = fmaf(y0, y0, fmaf(y1, y1, ss));
        }
      }
    ss += __shfl_xor(ss, 32);
    inv = 1.0f / sqrtf(ss * (1.0f / 128) + eps);
  }
#pragma unroll
  for (int qq = 0; qq < 2; ++qq)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 b0 = *reinterpret_cast<const f32x4*>(bsh + 32 * qq + 8 * g);
      const f32x4 b1 = *reinterpret_cast<const f32x4*>(bsh + 64 + 32 * qq + 8 * g);
      float p0[4], p1[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        p0[u] = fmaf(acc[m][qq][4 * g + u], scale, b0[u]);
        p1[u] = fmaf(acc[m][qq + 2][4 * g + u], scale, b1[u]);
      }
      if (KN) {
        const f32x4 w0 = *reinterpret_cast<const f32x4*>(knh + 32 * qq + 8 * g);
        const f32x4 w1 = *reinterpret_cast<const f32x4*>(knh + 64 + 32 * qq + 8 * g);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          p0[u] *= inv * w0[u];
          p1[u] *= inv * w1[u];
        }
      }
      if (ROT) {
        f32x4 cv, sv;
        rope_cs(L, st0 + (2 * L.wr + m) * 128, st1, qq, g, cv, sv);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float x0 = p0[u], x1 = p1[u];
          p0[u] = fmaf(x0, cv[u], -x1 * sv[u]);
          p1[u] = fmaf(x1, cv[u], x0 * sv[u]);
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) keep[qq][g][u] = p1[u];
      v0[qq][g] = make_uint2(pack2(p0[0], p0[1]), pack2(p0[2], p0[3]));
    }
  SB();
#pragma unroll
  for (int ph = 0; ph < 2; ++ph) {
#pragma unroll
    for (int qq = 0; qq < 2; ++qq)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int c = 4 * qq + g;
        const uint2 v = ph == 0 ? v0[qq][g]
                                : make_uint2(pack2(keep[qq][g][0], keep[qq][g][1]),
                                             pack2(keep[qq][g][2], keep[qq][g][3]));
        stg_write8(lds_addr(stg + rr * 64 + ((c ^ ((rr >> 1) & 7)) * 8) + (L.lane >> 5) * 4), v);
      }
    uint32_t ra[4];
    u32x4 rv[4];
#pragma unroll
    for (int pp = 0; pp < 4; ++pp) {
      const int ch = L.lane + 64 * pp;
      const int r2 = ch >> 3, c = ch & 7;
      ra[pp] = lds_addr(stg + r2 * 64 + ((c ^ ((r2 >> 1) & 7)) * 8));
    }
    stg_read4x16(ra, rv);
#pragma unroll
    for (int pp = 0; pp < 4; ++pp) {
      const int ch = L.lane + 64 * pp;
      const int r2 = ch >> 3, c = ch & 7;
      const u32x4 v = rv[pp];
      const int jj = j0 + 64 * L.wr + 32 * m + r2;
      const int off = jj < Tr ? (int)(jj * r_st * 2) + 128 * ph + c * 16 : (int)0x80000000;
      __builtin_amdgcn_raw_buffer_store_b128(v, rR, off, 0, 2);  // non-temporal: not read again here
    }
    SB();
  }
}

template <bool ROT, bool KN>
FI void epilogue(const Lane& L0, const f32x16 (&acc)[kMB][4], int j0, int Tr, long long r_st,
                 const float* bias_base, float scale, const float* kn_base, float eps,
                 uint16_t* stg, __amdgpu_buffer_rsrc_t rR, const float* st0, const float* st1) {
  // lane-derived addresses are formed here, inside the work-item loop, so that
  // they are not hoisted out of it and held across the k-loop
  Lane L = L0;
  L.lane = opaque(L0.lane);
  L.hi4 = 4 * (L.lane >> 5);
  const float* bsh = bias_base + 128 * L.wc + L.hi4;
  const float* knh = kn_base + L.hi4;
  epi_block<ROT, KN, 0>(L, acc, j0, Tr, r_st, bsh, scale, knh, eps, stg, rR, st0, st1);
  epi_block<ROT, KN, 1>(L, acc, j0, Tr, r_st, bsh, scale, knh, eps, stg, rR, st0, st1);
}

// KN: the receiver key norm is on (keys of calls that pass its weights); a
// separate instantiation keeps its registers out of the common kernel.
template <bool KN>
__global__ __launch_bounds__(512, 1) void staged_gemm_kernel(const TransferArgs p) {
  __shared__ __attribute__((aligned(1024))) unsigned char s0[32768];
  __shared__ __attribute__((aligned(1024))) unsigned char s1[32768];
  __shared__ __attribute__((aligned(1024))) unsigned char s2[32768];
  __shared__ __attribute__((aligned(1024))) unsigned char s3[32768];
  __shared__ __attribute__((aligned(1024))) float sbias[2 * 256];  // double-buffered tile bias
  __shared__ __attribute__((aligned(1024))) float skn[2 * 128];    // double-buffered key-norm weights
  __shared__ __attribute__((aligned(1024))) float st1[32 * 128];   // RoPE rows 0..31, swizzled
  __shared__ __attribute__((aligned(1024))) float st0[8 * 128];    // RoPE rows of the 8 block bases

  Lane L;
  L.lane = threadIdx.x & 63;
  L.wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  L.wr = L.wave >> 1;
  L.wc = L.wave & 1;
  L.hi4 = 4 * (L.lane >> 5);
  L.vw = L.lane * 16;
  {
    // feature DMA: block 2 wave + i holds rows 16 (2 wave + i) .. +16; lane l
    // fills row 16 blk + (l >> 2), slot l & 3, with chunk (l & 3) ^ sw(row)
    const int r_l = 32 * L.wave + (L.lane >> 2);
    L.vt0 = r_l * 64 + (((L.lane & 3) ^ sw(r_l)) * 16);
    L.vt1 = r_l * 64 + (((L.lane & 3) ^ sw(r_l + 16)) * 16);  // the block's 1 KB step is in soffset
    const int xr0 = 64 * L.wr + (L.lane & 31);
    L.xo0 = kWSt + xr0 * 64 + (((L.lane >> 5) ^ sw(xr0)) * 16);
    L.xo1 = kWSt + xr0 * 64 + (((2 + (L.lane >> 5)) ^ sw(xr0)) * 16);
    L.wo = L.wc * 4096 + L.lane * 16;
  }
  const int xcd = blockIdx.x & 7, wl = blockIdx.x >> 3, nwl = gridDim.x >> 3;
  const int n_quads = 2 * p.L_r * p.n_rt;
  const int n_jobs = 4 * ((n_quads - xcd + 7) / 8);  // this XCD's work items
  int jj = wl;
  if (jj >= n_jobs) return;
  const int KT = p.n_taps * (1024 / kBK);  // a multiple of 32
  const int wbytes = p.n_taps * 64 * 32 * 1024;
  const bool rope = p.rot && p.cs_r;

  Job J = decode(p, xcd, jj);
  dma_all(L, J, wbytes, 0, s0);
  dma_all(L, J, wbytes, 1, s1);
  dma_all(L, J, wbytes, 2, s2);
  auto dma_bias = [&](const Job& T, int half) {  // and the key-norm weights
    if (L.wave == 0 && T.bias)
      __builtin_amdgcn_global_load_lds(T.bias + L.lane * 4, (lds_void_t*)(sbias + half * 256), 16, 0, 0);
    if (KN && L.wave == 1 && T.keys && L.lane < 32)
      __builtin_amdgcn_global_load_lds(p.k_norm + T.l * 128 + L.lane * 4, (lds_void_t*)(skn + half * 128),
                                       16, 0, 0);
  };
  dma_bias(J, 0);
  if (!p.bias) sbias[threadIdx.x] = 0.0f;
  if (rope) {  // 32 rows of cos | sin for positions 0..31: 2 copies of 2 rows per wave
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = 2 * (2 * L.wave + i) + (L.lane >> 5);
      __builtin_amdgcn_global_load_lds(p.cs_t1 + r * 128 + (((L.lane & 31) ^ r) << 2),
                                       (lds_void_t*)(st1 + (2 * L.wave + i) * 256), 16, 0, 0);
    }
  }
  __builtin_amdgcn_s_waitcnt(0);
  f32x16 acc[kMB][4];  // set by each work item's first k-step
  bf16x8 f0x[kMB], f0w[4];
  __builtin_amdgcn_s_barrier();
  rd_frags(L, s0, 0, f0x, f0w);
  int tloc = 0;

  for (;;) {
    const int jn = jj + nwl;
    const bool has_next = jn < n_jobs;
    // the last job of the workgroup loads its own first k-tiles once more into
    // stages nothing reads again, so every k-tile issues the same loads (the
    // index is chosen, not the decoded item, which keeps N in registers)
    const Job N = decode(p, xcd, has_next ? jn : jj);
    const bool rot = rope && J.keys;
    if (rot && L.wave < 4) {  // RoPE rows of this tile's 32-row block bases (rows 2 w, 2 w + 1)
      const int jb = min(J.j0 + 64 * L.wave + 32 * (L.lane >> 5), J.Tr - 1);
      __builtin_amdgcn_global_load_lds(p.cs_r + (long long)(J.pos0 + jb) * 128 + (L.lane & 31) * 4,
                                       (lds_void_t*)(st0 + 2 * L.wave * 128), 16, 0, 0);
    }
    // k-tiles 0..3 (k-tile 0 landed before the previous item's epilogue)
    ktile<20, true>(L, acc, f0x, f0w, true, s0, s1, s3, J, wbytes, 3);
    ktile<20, false>(L, acc, f0x, f0w, true, s1, s2, s0, J, wbytes, 4);
    ktile<4, false>(L, acc, f0x, f0w, true, s2, s3, s1, J, wbytes, 5);
    ktile<4, false>(L, acc, f0x, f0w, true, s3, s0, s2, J, wbytes, 6);
    for (int kt = 4; kt < KT - 4; kt += 4) {
      ktile<4, false>(L, acc, f0x, f0w, true, s0, s1, s3, J, wbytes, kt + 3);
      ktile<4, false>(L, acc, f0x, f0w, true, s1, s2, s0, J, wbytes, kt + 4);
      ktile<4, false>(L, acc, f0x, f0w, true, s2, s3, s1, J, wbytes, kt + 5);
      ktile<4, false>(L, acc, f0x, f0w, true, s3, s0, s2, J, wbytes, kt + 6);
    }
    // the last 4 k-tiles: this job's last one, then the next job's first three
    ktile<4, false>(L, acc, f0x, f0w, true, s0, s1, s3, J, wbytes, KT - 1);
    ktile<4, false>(L, acc, f0x, f0w, true, s1, s2, s0, N, wbytes, 0);
    ktile<4, false>(L, acc, f0x, f0w, true, s2, s3, s1, N, wbytes, 1);
    ktile<4, false>(L, acc, f0x, f0w, false, s3, s0, s2, N, wbytes, 2);
    // The wait at the start of the last k-tile left only the next job's k-tile
    // 1 loads outstanding, so this job's bias and RoPE rows and the next job's
    // k-tile 0 have landed; k-tiles 1 and 2 keep loading through the epilogue,
    // into stages the epilogue does not touch.
    __builtin_amdgcn_s_barrier();  // every wave is past its last read of stage 3
    {
      const __amdgpu_buffer_rsrc_t rR =
          mk_rsrc(J.rbase + (long long)L.wc * p.r_sh, (int)((long long)J.Tr * p.r_st * 2));
      uint16_t* stg = reinterpret_cast<uint16_t*>(s3) + L.wave * 32 * 64;  // stage 3 is free here
      const float* bias_base = sbias + (tloc & 1) * 256;
      const float* kn_base = skn + (tloc & 1) * 128;
      const float eps = p.k_norm_eps;
      // With concatenated taps the slabs are shared by receiver layers with
      // different r, so 1/r scales the product A x_j (equal to A (x_j / r));
      // the interpolating build already scaled x_j.
      const float scale = (p.inv_r && p.concat) ? p.inv_r[J.l * 2 + (J.keys ? 0 : 1)] : 1.0f;
      if (KN && J.keys) {
        if (rot) epilogue<true, true>(L, acc, J.j0, J.Tr, p.r_st, bias_base, scale, kn_base, eps, stg, rR, st0, st1);
        else epilogue<false, true>(L, acc, J.j0, J.Tr, p.r_st, bias_base, scale, kn_base, eps, stg, rR, st0, st1);
      } else {
        if (rot) epilogue<true, false>(L, acc, J.j0, J.Tr, p.r_st, bias_base, scale, kn_base, eps, stg, rR, st0, st1);
        else epilogue<false, false>(L, acc, J.j0, J.Tr, p.r_st, bias_base, scale, kn_base, eps, stg, rR, st0, st1);
      }
    }
    if (!has_next) break;
    // The next job's bias goes into the other half of sbias only now: a load
    // into LDS issued before the epilogue's LDS reads would make them wait for
    // every load in flight, the next job's k-tiles 1 and 2 included.
    dma_bias(N, (tloc + 1) & 1);
    __builtin_amdgcn_s_barrier();  // staging in stage 3 is read
    rd_frags(L, s0, 0, f0x, f0w);
    jj = jn;
    J = N;
    ++tloc;
  }
  __builtin_amdgcn_s_waitcnt(0);  // no load into LDS outlives the workgroup
}

}  // namespace

hipError_t launch_staged_gemm(const TransferArgs& a, hipStream_t s) {
  if (a.n_rt < 1 || a.L_r < 1) return hipSuccess;
  if (!a.xs || a.H_r != 8 || a.H_s != 8 || a.d_h != 128) return hipErrorInvalidValue;
  int dev = 0, n_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const int grid = 8 * std::max(1, n_cu / 8);  // whole XCD rounds: workgroup i runs on XCD i % 8
  if (a.k_norm) hipLaunchKernelGGL(staged_gemm_kernel<true>, dim3((unsigned)grid), dim3(512), 0, s, a);
  else hipLaunchKernelGGL(staged_gemm_kernel<false>, dim3((unsigned)grid), dim3(512), 0, s, a);
  return hipGetLastError();
}

}  // namespace hf
