// Internal interface between the C-ABI layer (abi.cpp) and the kernel files.
// Plain structs passed by value as kernel arguments (kept under 4 KB).
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

#include "heterofold.h"

namespace hf {

constexpr int kAlignBlock = 256;  // receiver rows per alignment workgroup
constexpr int kRopeDeltaRows = 16;  // sender RoPE table rows the bf16 kernels always read
constexpr uint32_t kPackedMagic = 0x4B504648u;  // "HFPK": first word of a packed map buffer

struct AlignArgs {
  const int32_t* s_beg;
  const int32_t* s_end;
  const int32_t* r_beg;
  const int32_t* r_end;
  int32_t* row_ptr;
  int32_t* col;
  int32_t* num;
  int32_t* den;
  long long* blk_sum;   // [nblk] entries counted by each workgroup
  long long* blk_off;   // [nblk] exclusive prefix of blk_sum
  int32_t* blk_last;    // [nblk] last TA partner found in the workgroup, -1 if none
  int32_t* blk_carry;   // [nblk] TA partner carried into the workgroup
  long long cap;        // entries the col/num buffers hold
  int32_t mode;
  int32_t B;
  int32_t nblk;
  int32_t total_rows;
  int32_t blk_start[HF_MAX_BATCH + 1];  // first workgroup of each sequence
  int32_t s0[HF_MAX_BATCH];             // first sender span of each sequence
  int32_t Ts[HF_MAX_BATCH];
  int32_t r0[HF_MAX_BATCH];             // first receiver span / CSR row of each sequence
  int32_t Tr[HF_MAX_BATCH];
};

// Workspace layout of the alignment: four arrays of nblk entries.
size_t align_workspace_bytes(int nblk);

struct TransferArgs {
  const void* S;        // sender cache
  void* R;              // receiver cache
  const void* Wp;       // packed maps (past the header)
  const float* bias;    // [L_r][2][d_r] or nullptr
  const int32_t* row_ptr;
  const int32_t* col;
  const int32_t* num;
  const int32_t* den;
  const int32_t* tile_rec;  // per-row-tile staging records (tiled bf16 kernel)
  int32_t* work_ctr;        // next work item of the persistent tiled kernel
  int32_t n_wg;             // workgroups of the persistent tiled kernel
  const float* cs_s;    // sender RoPE table [P_s][d_h]: cos of the d_h/2 angles, then sin
  const float* cs_r;    // receiver RoPE table [P_r][d_h], same layout
  const float* inv_r;   // [L_r][2] scalar 1/r per layer and role, or nullptr (1)
  const float* k_norm;  // [L_r][d_h] receiver key RMSNorm weights, or nullptr
  float k_norm_eps;
  long long s_sb, s_sl, s_sc, s_sh, s_st;
  long long r_sb, r_sl, r_sc, r_sh, r_st;
  int32_t L_r, H_s, H_r, d_h;
  int32_t unrot, rot;       // RoPE on keys: un-rotate sender / rotate receiver
  int32_t s_extent;         // bytes spanned by one (sequence, layer, role) slab of the
                            // sender cache; 0 if that is 2^31 or more
  int32_t B;
  int32_t rows_per_tile;
  int32_t tiles_per_lc;     // row tiles of one (layer, role), summed over the batch
  int32_t tile_start[HF_MAX_BATCH + 1];
  int32_t Ts[HF_MAX_BATCH];
  int32_t Tr[HF_MAX_BATCH];
  int32_t row0[HF_MAX_BATCH];    // first CSR row of each sequence
  int32_t pos0_s[HF_MAX_BATCH];
  int32_t pos0_r[HF_MAX_BATCH];
  int32_t n_taps;           // sender layers per receiver layer whose features are concatenated
  int32_t concat;           // 1: taps[l][0..n_taps) each with weight 1; 0: interpolate lo, hi
  uint8_t lo[HF_MAX_LAYERS];
  uint8_t hi[HF_MAX_LAYERS];
  uint8_t taps[HF_MAX_LAYERS][3];
  float wlo[HF_MAX_LAYERS];
  float whi[HF_MAX_LAYERS];
  // Staged path (bf16, 8 sender and 8 receiver heads of 128): the build writes
  // the aligned features of every slab -- (role, receiver layer) for the
  // interpolating map, (role, sender layer) for concatenated taps -- into xs,
  // and the GEMM reads them back.  Slab layout: [256-row tile][32-feature
  // k-tile][256 rows][32] bf16, sequences padded to whole 256-row tiles.
  uint16_t* xs;            // nullptr: fused path
  long long xs_slab;       // elements per slab
  int32_t n_slab_layers;   // L_r (interpolating map) or sender layers (taps)
  int32_t n_rt;            // 256-row tiles of the batch
  int32_t rt_start[HF_MAX_BATCH + 1];  // first 256-row tile of each sequence
  const float* cs_t1;      // receiver RoPE rows of positions 0..31 (cos | sin)
};
static_assert(sizeof(TransferArgs) <= 4096, "kernel argument size");

// Staged path: the shapes it serves, its slab and table bytes, and its launches.
bool staged_supported(int dtype, int H_s, int H_r, int d_h);
constexpr int kStagedRows = 256;   // rows per GEMM tile
constexpr size_t kStagedT1Bytes = 32 * 128 * 4;
hipError_t launch_staged_build(const TransferArgs& a, hipStream_t s);
hipError_t launch_staged_gemm(const TransferArgs& a, hipStream_t s);

// Rows per workgroup tile of the transfer kernels.
int transfer_rows_per_tile(int dtype, int H_r, int H_s, int n_taps, int d_h);
// Device bytes of the staging record each row tile needs (0 where the kernel
// that runs keeps no records), and the launch that writes the records
// (a.tile_rec, one per tile of the batch) before launch_transfer.
size_t transfer_tile_record_bytes(int dtype, int H_r, int H_s, int d_h);
// Workgroups of the persistent tiled kernel on a device with n_cu compute units.
int transfer_persistent_grid(const TransferArgs& a, int n_cu);
hipError_t launch_transfer_stage(int dtype, const TransferArgs& a, hipStream_t s);

hipError_t launch_alignment(const AlignArgs& a, hipStream_t s);
hipError_t launch_rope_table(float* tab, int P, int d_h, double theta, hipStream_t s);
// Writes the header and the packed maps (A_packed: hf_packed_maps_bytes bytes).
hipError_t launch_pack_maps(int dtype, int n_lc, int d_r, int d_in, const void* A, void* A_packed,
                            hipStream_t s);
hipError_t launch_transfer(int dtype, const TransferArgs& a, hipStream_t s);
// Device address of the no-allocation scratch (HF_NOALLOC_SCRATCH_BYTES) on the
// current device; resolved once per device.
hipError_t noalloc_scratch(void** ptr);

// Offline map construction (fp64).  Workspace layouts are private to recolor.hip.
int moments_chunks(long long n);
size_t recolor_moments_workspace_bytes(long long n, int p, int q);
// Weight sum, r, means of [x/r | y] and the centring shifts (kept in the workspace).
hipError_t launch_recolor_stats(int dtype, long long n, int p, int q, const void* X,
                                long long ldx, const void* Y, long long ldy, const float* w,
                                double* r, double* mu, void* workspace, hipStream_t s);
// Partial Gram tiles of the centred samples, from the shifts launch_recolor_stats
// left in the workspace; then their fixed-order sum into the joint covariance.
hipError_t launch_recolor_cov(int dtype, long long n, int p, int q, const void* X, long long ldx,
                              const void* Y, long long ldy, const float* w, void* workspace,
                              hipStream_t s);
hipError_t launch_recolor_cov_reduce(long long n, int p, int q, double* cov, void* workspace,
                                     hipStream_t s);
size_t recolor_solve_workspace_bytes(int p, int q);
hipError_t launch_recolor_solve(int p, int q, const double* mu, const double* cov, double lam,
                                double* A, double* b, hf_recolor_info* info, void* workspace,
                                hipStream_t s);
size_t fold_workspace_bytes(int p, int rank);
hipError_t launch_fold(int p, int q, int rank, const double* A, const double* b, const double* B,
                       const double* G, double* A_out, double* b_out, void* workspace,
                       hipStream_t s);
hipError_t launch_gemm_f64(int m, int n, long long k, const double* A, long long lda, int ak,
                           const double* B, long long ldb, int bk, double* D, long long ldd,
                           double alpha, double beta, const double* C, long long ldc,
                           double gamma, hipStream_t s);

}  // namespace hf
