/*
 * heterofold.h -- C ABI of the HeteroFold transfer-time path on AMD MI355X
 * (gfx950).
 *
 * The path turns a frozen sender model's KV cache into a frozen receiver
 * model's KV cache without running the receiver's prefill (Sec. 3, opening
 * paragraph: map C_S(x) to a receiver-compatible cache).  It has four steps:
 *
 *   1. hf_build_alignment  -- which sender tokens each receiver token reads,
 *      from the two tokenizers' character spans (Sec. 3.1 "Token Alignment";
 *      App. B.1), as a CSR span table.
 *   2. hf_build_layer_map  -- which sender layers feed each receiver layer
 *      (hf_build_layer_taps: the paper's three-layer neighbourhood).
 *   3. hf_transfer_kv      -- gather, segment-mean and layer-interpolate the
 *      sender cache, un-rotate post-RoPE sender keys, apply the folded affine
 *      map y = A x + b of each receiver layer and role (Eq. 9), rotate keys at
 *      the receiver's positions, and write the receiver cache.
 *   4. (RoPE un-rotation / re-rotation is fused into step 3.)
 *
 * hf_pack_maps re-lays the static maps out once for the matrix-core kernel.
 *
 * Conventions for every call:
 *  - Returns HF_OK (0) or a negative hf_status; hf_last_error() then holds a
 *    thread-local description.  Nothing aborts and no C++ exception crosses
 *    the ABI.
 *  - "device" pointers are HIP device memory owned by the caller; "host"
 *    pointers are host memory owned by the caller and read only during the
 *    call.  The library allocates no device memory; scratch space comes from a
 *    caller workspace whose size a *_workspace_bytes query gives.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and
 *    runs asynchronously; no call synchronizes the host (the profiler query
 *    excepted).  Launch errors are reported as HF_ERR_HIP.
 *  - All host-checkable arguments are validated before anything is launched.
 *    Device-side data that cannot be checked on the host (character offsets,
 *    CSR contents) never causes an out-of-bounds access: indices are clamped
 *    into the buffers the sizes describe.  The one exception is the CSR row
 *    offsets the transfer calls read, which they trust: they must be the table
 *    hf_build_alignment wrote (always monotone and within its capacity).
 *  - Character spans: token t of a sequence covers characters [beg[t], end[t]).
 *    Valid spans are sorted and non-overlapping: 0 <= beg[t] <= end[t] <=
 *    beg[t+1].  Empty tokens (beg == end) and gaps are allowed.  Results for
 *    spans that break this rule are unspecified but memory-safe.
 */
#ifndef HETEROFOLD_H
#define HETEROFOLD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HF_VERSION 2
#define HF_MAX_BATCH 64   /* sequences per call */
#define HF_MAX_LAYERS 128 /* receiver layers per call */

typedef enum {
  HF_OK = 0,
  HF_ERR_NULL = -1,        /* a required pointer is NULL */
  HF_ERR_SHAPE = -2,       /* sizes, strides or counts are inconsistent */
  HF_ERR_OFFSETS = -3,     /* character spans break the sorted/non-overlapping rule (host check) */
  HF_ERR_MODE = -4,        /* unknown alignment or layer mode */
  HF_ERR_DTYPE = -5,       /* unknown or mismatched storage type */
  HF_ERR_CAPACITY = -6,    /* an output or workspace buffer is too small */
  HF_ERR_HIP = -7,         /* a HIP runtime call or kernel launch failed */
  HF_ERR_UNSUPPORTED = -8  /* a valid shape the library has no kernel for */
} hf_status;

typedef enum { HF_ALIGN_OVERLAP = 0, HF_ALIGN_TA = 1 } hf_align_mode;
typedef enum { HF_LAYERS_INTERP2 = 0 } hf_layer_mode;
typedef enum { HF_F32 = 0, HF_BF16 = 1 } hf_dtype;

/*
 * Optional parts of the paper's cache construction for hf_transfer_kv and
 * hf_transfer_kv_taps (pass NULL for none of them):
 *   inv_r      device fp32 [L_r][2] or NULL: the scalar 1/r of Eq. 3 per
 *              receiver layer and role; the map sees x_j / r (Eq. 9).  The
 *              scaling happens in fp32 before x_j is rounded.  NULL: 1 (r
 *              folded into A by the caller).
 *   k_norm     device fp32 [L_r][d_h] or NULL: the receiver's key
 *              normalization (App. B.1: mapped keys go through the receiver's
 *              own key normalization, then its RoPE).  Per receiver head of
 *              d_h features: y <- y / sqrt(mean(y^2) + k_norm_eps) * k_norm[l],
 *              after the bias and before the receiver rotation.  Keys only.
 *   k_norm_eps epsilon under the root, finite and >= 0.
 * Buffers are caller-owned and 4-byte aligned.
 */
typedef struct {
  const float* inv_r;
  const float* k_norm;
  float k_norm_eps;
} hf_transfer_opts;

/* Thread-local text of the last failure of a call made on this thread. */
const char* hf_last_error(void);
int32_t hf_version(void);

/* ------------------------------------------------------------------------ */
/* Step 1: cross-tokenizer alignment (Sec. 3.1 "Token Alignment"; App. B.1). */
/* ------------------------------------------------------------------------ */

/*
 * Entries the col / num buffers of hf_build_alignment must hold for valid
 * spans of B sequences: the sum over sequences of T_s + 2 T_r in
 * HF_ALIGN_OVERLAP mode (a receiver row reads the sender tokens its span
 * overlaps: with both tokenizations tiling one text, the distinct boundaries
 * of the two, at most T_s + T_r; plus one fallback entry per empty or
 * uncovered row), and of T_r in HF_ALIGN_TA mode (one entry per row).
 * s_len, r_len: host int32 [B] sender / receiver token counts.
 * Returns -1 (and sets hf_last_error) on bad arguments.
 */
int64_t hf_alignment_nnz_capacity(int32_t B, const int32_t* s_len, const int32_t* r_len,
                                  int32_t mode);

/* Workspace bytes hf_build_alignment needs for this batch. */
size_t hf_alignment_workspace_bytes(int32_t B, const int32_t* r_cu);

/*
 * Build the alignment table of B independent sequences.
 *
 * Inputs
 *   s_cu, r_cu        host int32 [B+1]: prefix sums of token counts.  A
 *                     sequence with T_r > 0 needs T_s > 0.
 *   s_beg, s_end      device int32 [s_cu[B]]: sender spans, sequences back to back.
 *   r_beg, r_end      device int32 [r_cu[B]]: receiver spans.
 *   mode              HF_ALIGN_TA: the paper's Token Alignment.  Nonempty
 *                     sender and receiver tokens that end at the same character
 *                     are paired (the largest such sender index); other
 *                     receiver tokens take the sender token of the latest
 *                     preceding shared boundary, or the first nonempty sender
 *                     token before any (index 0 if none is nonempty).  One
 *                     entry per row, weight 1.
 *                     HF_ALIGN_OVERLAP: receiver token j reads every sender
 *                     token i whose span overlaps its own, with weight
 *                     num/den_j where num = shared characters and den_j = their
 *                     sum; a row with no overlap holds its TA entry (weight 1).
 * Outputs (device, caller-allocated)
 *   row_ptr  int32 [r_cu[B]+1]  global CSR row offsets; row r_cu[b]+j is
 *                               receiver token j of sequence b.
 *   col      int32 [nnz_capacity]  sender token index, local to the sequence.
 *   num      int32 [nnz_capacity]  weight numerator (1 in TA mode).
 *   den      int32 [r_cu[B]]       weight denominator of the row.
 *   Entries of a row are in ascending col order.  For valid spans the table
 *   is unique and the result is bit-exact.
 * nnz_capacity must be >= hf_alignment_nnz_capacity() for the same lengths
 * and mode; otherwise HF_ERR_CAPACITY.  (Spans that break the validity rule may need more; the
 * kernels then drop entries past the capacity and clamp row_ptr to it.)
 * workspace: device, >= hf_alignment_workspace_bytes() bytes, 16-B aligned.
 */
int32_t hf_build_alignment(int32_t B, const int32_t* s_cu, const int32_t* r_cu,
                           const int32_t* s_beg, const int32_t* s_end,
                           const int32_t* r_beg, const int32_t* r_end, int32_t mode,
                           int32_t* row_ptr, int32_t* col, int32_t* num, int32_t* den,
                           int64_t nnz_capacity, void* workspace, size_t workspace_bytes,
                           void* stream);

/* Host check of one sequence's spans against the validity rule above:
 * HF_OK or HF_ERR_OFFSETS (HF_ERR_NULL / HF_ERR_SHAPE for bad arguments). */
int32_t hf_validate_offsets_host(int32_t T, const int32_t* beg, const int32_t* end);

/* ------------------------------------------------------------------------ */
/* Step 2: layer map.                                                        */
/* ------------------------------------------------------------------------ */

/*
 * HF_LAYERS_INTERP2: receiver layer j (0-based) sits at sender depth
 * p = j (L_s-1)/(L_r-1) and linearly interpolates sender layers lo = floor(p)
 * and hi = min(lo+1, L_s-1) with weights (den-rem)/den and rem/den, where
 * rem/den = p - lo exactly (rem == 0: a single tap).  L_r == 1 gives
 * (0, 0, 0, 1).  Outputs are host int32 [L_r] each.  Pure host code.
 * (The paper's own map feeds three sender layers at offsets -4, 0, +4 around
 * a proportional depth, Eq. 1; this interpolating map is the two-tap variant.)
 */
int32_t hf_build_layer_map(int32_t L_s, int32_t L_r, int32_t mode, int32_t* lo, int32_t* hi,
                           int32_t* rem, int32_t* den);

/*
 * The paper's own layer alignment (Sec. 3.1 "Layer Alignment", Eq. 1),
 * 0-based: receiver layer j is matched to sender layer
 * pi(j) = round(j (L_s-1)/(L_r-1)) (exact rational, ties to even; L_r == 1
 * gives 0) and reads the three sender layers clip(pi-4, pi, pi+4) to
 * [0, L_s-1].  taps: host int32 [L_r][3], caller-owned.  Pure host code.
 * Feed the table to hf_transfer_kv_taps with n_taps = 3.
 * Errors: HF_ERR_SHAPE (L_s < 1 or L_r < 1), HF_ERR_NULL.
 */
int32_t hf_build_layer_taps(int32_t L_s, int32_t L_r, int32_t* taps);

/* ------------------------------------------------------------------------ */
/* Step 3: KV transfer.                                                      */
/* ------------------------------------------------------------------------ */

/*
 * A KV cache in device memory.  Element (b, l, c, h, t, e) -- sequence b,
 * layer l, role c (0 = K, 1 = V), KV head h, token t, channel e -- lives at
 * ptr + b*stride_b + l*stride_l + c*stride_c + h*stride_h + t*stride_t + e
 * (strides in elements; channels contiguous).  The canonical layout
 * [B][L][2][H][T_cap][d_h] is the receiver cache layout [L,2,H_kv,T,d_h] per
 * sequence; any other order of the strides works the same way (token-major
 * storage [T][H], rows padded past d_h, a cache inside a larger buffer).
 * ptr and every stride must keep rows 16-byte aligned.  A receiver whose rows
 * overlap gets racing writes.
 */
typedef struct hf_kv_desc {
  void* ptr;
  int32_t dtype; /* hf_dtype */
  int32_t L, H, d_h, T_cap;
  int64_t stride_b, stride_l, stride_c, stride_h, stride_t;
} hf_kv_desc;

/*
 * Rotary position embedding (rotate-half: channel k pairs with k + d_h/2,
 * angle pos * theta^(-2k/d_h)).  Sender token i sits at pos0_s[b] + i and
 * receiver token j at pos0_r[b] + j (host int32 [B], NULL = 0).  If
 * unrotate_sender_k, the stored sender keys are post-RoPE and are un-rotated
 * at sender positions with theta_s before mapping; if rotate_receiver_k the
 * mapped keys are rotated at receiver positions with theta_r (the receiver
 * applies its own RoPE to mapped keys: Sec. 3.3 "Folding for inference";
 * App. B.1).  Angles are formed in fp64; the rotation runs in fp32.
 */
typedef struct hf_rope {
  double theta_s, theta_r;
  int32_t unrotate_sender_k, rotate_receiver_k;
  const int32_t* pos0_s;
  const int32_t* pos0_r;
} hf_rope;

/* Bytes of a packed map buffer for L_r receiver layers, 2 roles, d_r x d_in:
 * an HF_PACKED_HEADER_BYTES header (what was packed) followed by the maps in
 * fragment order, so it is larger than the unpacked maps.  0 on bad arguments. */
#define HF_PACKED_HEADER_BYTES 256
size_t hf_packed_maps_bytes(int32_t L_r, int32_t d_r, int32_t d_in, int32_t dtype);

/*
 * Re-lay the folded maps out for hf_transfer_kv.  A: device [L_r][2][d_r][d_in]
 * row-major in `dtype` (row n maps the flattened sender feature, head-major
 * index h*d_h + e, to receiver feature n = h'*d_h + e'; this is the transpose
 * of the paper's row-vector A_final of Eq. 9, with the scalar 1/r of Eq. 3
 * already folded in).  A_packed: device, hf_packed_maps_bytes() bytes,
 * 16-B aligned, not overlapping A; it receives a header (the word "HFPK",
 * layout version, dtype, L_r, d_r, d_in) and the maps re-laid out in the
 * matrix-core fragment order the bf16 kernels read (fp32 maps are copied
 * row-major).  Maps are static, so this runs once per model pair.  bf16 needs
 * d_in % 16 == 0 and d_r % 32 == 0.
 */
int32_t hf_pack_maps(int32_t L_r, int32_t d_r, int32_t d_in, int32_t dtype, const void* A,
                     void* A_packed, void* stream);

/*
 * Workspace bytes hf_transfer_kv and hf_transfer_kv_taps need: the RoPE
 * cos/sin tables (none without RoPE) and, for bf16 with 4 or 8 receiver heads
 * and at most 8 sender heads, an 8 KB staging record per 64-row receiver tile
 * (the tile's alignment entries, written once per call and read by every
 * receiver layer and role) plus 256 bytes for a work counter.  0 when neither
 * applies.  Calls that share a workspace must not overlap.
 */
size_t hf_transfer_workspace_bytes(int32_t B, const int32_t* s_len, const int32_t* r_len,
                                   const hf_kv_desc* sender, const hf_kv_desc* receiver,
                                   const hf_rope* rope);

/*
 * Workspace bytes for the staged path of hf_transfer_kv (n_taps = 0) or
 * hf_transfer_kv_taps (n_taps = 1..3): hf_transfer_workspace_bytes() plus a
 * 16 KB table and one slab of aligned features per (role, receiver layer) for
 * the interpolating map, or per (role, sender layer) for concatenated taps,
 * each slab 2 bytes x 1024 features x the batch's receiver rows rounded up to
 * 256 per sequence (about 61 MB per slab for one 29K-row sequence).  0 where
 * the staged path does not apply: it serves bf16 with 8 sender and 8 receiver
 * heads of d_h = 128.
 * The transfer calls take the staged path when their workspace holds at least
 * this many bytes, the shape is served, and every sequence's receiver rows
 * span less than 2 GiB of its cache (the multiply addresses them with 32-bit
 * byte offsets); otherwise the fused path.  Both compute the same values up to
 * rounding: the staged path builds x_j as the fused path does (one bf16
 * rounding), stores it, and multiplies it in a separate kernel whose epilogue
 * applies the bias, the key norm and the receiver RoPE.  One difference in
 * where rounding happens: with concatenated taps the slabs are shared by
 * receiver layers with different r, so the staged path rounds x_j without
 * 1/r and scales the product A x_j by 1/r in fp32, where the fused path
 * rounds x_j / r (equal in exact arithmetic).  hf_transfer_kv_noalloc always
 * takes the fused path.
 */
size_t hf_transfer_staged_workspace_bytes(int32_t B, const int32_t* s_len, const int32_t* r_len,
                                          const hf_kv_desc* sender, const hf_kv_desc* receiver,
                                          const hf_rope* rope, int32_t n_taps);

/*
 * Map the sender caches of B sequences to receiver caches.  For receiver
 * layer l, role c and receiver token j of sequence b:
 *   m_i = a_lo S[lo_l, c, :, i, :] + a_hi S[hi_l, c, :, i, :]      (layer map)
 *   u_i = U_s(pos0_s + i) m_i  for keys when rope->unrotate_sender_k, else m_i
 *   x_j = sum over row j of (num/den_j) u_i, flattened head-major   (alignment)
 *   y_j = A[l, c] (x_j * inv_r[l, c]) + bias[l, c]                  (Eq. 9)
 *   keys: RMSNorm per receiver head when opts->k_norm (App. B.1), then
 *         y_j <- R_r(pos0_r + j) y_j per receiver head when rotate_receiver_k
 *   R[l, c, h', j, e'] = y_j[h'*d_h + e']
 * Arguments
 *   s_len, r_len   host int32 [B]: token counts (<= sender/receiver T_cap).
 *   row_ptr, col, num, den   device: the table hf_build_alignment wrote for
 *                  the same batch (row r_cu[b]+j as documented there).  col is
 *                  clamped into the sequence; row_ptr is trusted (see above).
 *   lo, hi, rem, den_l       host int32 [receiver->L]: hf_build_layer_map's table.
 *   sender, receiver         cache descriptors; same dtype and d_h.
 *                  receiver->L is L_r; d_in = sender->H*d_h, d_r = receiver->H*d_h.
 *   A_packed       device: maps packed by hf_pack_maps (same L_r, d_r, d_in, dtype).
 *   A_packed_bytes the size of that buffer; anything other than
 *                  hf_packed_maps_bytes(L_r, d_r, d_in, dtype) -- an unpacked map
 *                  [L_r][2][d_r][d_in] in particular -- returns HF_ERR_SHAPE.
 *   bias           device fp32 [L_r][2][d_r], or NULL for zero bias.
 *   rope           NULL = no RoPE.
 *   opts           NULL, or the optional 1/r and key normalization (above).
 *   workspace      device, >= hf_transfer_workspace_bytes(), 256-B aligned;
 *                  >= hf_transfer_staged_workspace_bytes(..., 0) selects the
 *                  staged path where it applies (see there).
 * Numerics: HF_F32 computes in fp32 throughout.  HF_BF16 forms x_j in fp32,
 * rounds it once to bf16 (round-to-nearest-even), multiplies on the matrix
 * cores with fp32 accumulation, adds bias and rotates in fp32, and rounds the
 * result once to bf16.
 * Supported by this library: d_h == 128 for HF_BF16 with receiver H in
 * {2, 4, 8} and one (layer, role) map under 2 GiB; any even d_h and H for
 * HF_F32 (d_in <= 4096).  Other valid shapes -- bf16 with d_h == 64 among
 * them -- return HF_ERR_UNSUPPORTED before anything is launched.
 * Receiver rows past r_len are not written.
 */
int32_t hf_transfer_kv(int32_t B, const int32_t* s_len, const int32_t* r_len,
                       const int32_t* row_ptr, const int32_t* col, const int32_t* num,
                       const int32_t* den, const int32_t* lo, const int32_t* hi,
                       const int32_t* rem, const int32_t* den_l, const hf_kv_desc* sender,
                       const hf_kv_desc* receiver, const void* A_packed, size_t A_packed_bytes,
                       const float* bias, const hf_rope* rope, const hf_transfer_opts* opts,
                       void* workspace, size_t workspace_bytes, void* stream);

/*
 * hf_transfer_kv for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation.
 * Arguments, results and errors as hf_transfer_kv, without the workspace: the
 * scratch it needs (the RoPE tables, one 8 KB staging record per 64-row
 * receiver tile, a work counter; hf_transfer_workspace_bytes gives the amount)
 * lives in a device array of HF_NOALLOC_SCRATCH_BYTES inside the library,
 * which each GPU the library runs on holds from load until the process ends.
 * A transfer that needs more returns HF_ERR_CAPACITY before anything is
 * launched (at 64 MiB: a 32K-token sequence needs about 34 MB, four of them
 * about 47 MB).  The call allocates nothing (no hipMalloc / hipFree, no
 * profiler events: its launches are not timed by hf_profiler_*); its first
 * call on a device resolves the array's device address.  Every call on one
 * GPU shares that GPU's array: calls that overlap on one GPU (different
 * streams, different host threads) race and must be serialized by the
 * caller.  Nothing in the array has to start at zero: each call writes what
 * it reads before reading it.
 */
#define HF_NOALLOC_SCRATCH_BYTES (64 << 20)
int32_t hf_transfer_kv_noalloc(int32_t B, const int32_t* s_len, const int32_t* r_len,
                               const int32_t* row_ptr, const int32_t* col, const int32_t* num,
                               const int32_t* den, const int32_t* lo, const int32_t* hi,
                               const int32_t* rem, const int32_t* den_l,
                               const hf_kv_desc* sender, const hf_kv_desc* receiver,
                               const void* A_packed, size_t A_packed_bytes, const float* bias,
                               const hf_rope* rope, const hf_transfer_opts* opts, void* stream);

/*
 * hf_transfer_kv for maps over concatenated sender layers (Sec. 3.1 Eq. 2,
 * with the folded map of Eq. 9): receiver layer l reads the n_taps sender
 * layers taps[l][0..n_taps) without interpolation, and its map sees their
 * aligned features side by side,
 *   x_j = [x_j^{t_1} | ... | x_j^{t_n}],
 *   x_j^t = sum over row j of (num/den_j) U_s(pos0_s + i) S[t, c, :, i, :]
 * (each block flattened head-major; U_s for keys when unrotate_sender_k).
 * Arguments as hf_transfer_kv, except
 *   n_taps     1..3 (3 for hf_build_layer_taps's table)
 *   taps       host int32 [receiver->L][n_taps], sender layers in [0, sender->L)
 *   A_packed   maps A[l, c] of shape [d_r][n_taps * d_in] packed by
 *              hf_pack_maps with its d_in argument = n_taps * sender->H * d_h;
 *              A_packed_bytes its size, checked as in hf_transfer_kv.
 * Shapes supported, numerics, ownership and errors as hf_transfer_kv; for
 * HF_F32 the limit is n_taps * d_in <= 4096.
 */
int32_t hf_transfer_kv_taps(int32_t B, const int32_t* s_len, const int32_t* r_len,
                            const int32_t* row_ptr, const int32_t* col, const int32_t* num,
                            const int32_t* den, int32_t n_taps, const int32_t* taps,
                            const hf_kv_desc* sender, const hf_kv_desc* receiver,
                            const void* A_packed, size_t A_packed_bytes, const float* bias,
                            const hf_rope* rope, const hf_transfer_opts* opts, void* workspace,
                            size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Offline construction of the maps (fp64, off the transfer path).           */
/* ------------------------------------------------------------------------ */
/*
 * For one receiver layer and role, N paired calibration samples x_n (aligned
 * sender feature, p = d~_S values: the concatenated taps of Eq. 2) and y_n
 * (receiver feature, q = d_R values) with weights w_n.  The three calls below
 * give the folded map the transfer calls take:
 *
 *   hf_recolor_moments  r of Eq. 3, and the weighted means and joint
 *                       covariance of [x/r | y] (Sec. 3.2);
 *   hf_recolor_solve    Recolor (Eq. 4-5): A = S_Z^{-1/2} R* S_Y^{1/2},
 *                       b = mu_Y - mu_Z A, R* = U Q^T from the thin SVD
 *                       S_Z^{-1/2} S_ZY S_Y^{-1/2} = U Lambda Q^T;
 *   hf_fold_map         the output-aware correction folded in (Eq. 9):
 *                       A (I + B G), b (I + B G).
 *
 * Maps are returned in the transfer path's orientation: A stored [q][p]
 * row-major (the paper's row-vector A transposed), so y = A (x/r) + b.  The
 * caller converts A to the storage type of hf_pack_maps, b to the fp32 bias,
 * and 1/r to hf_transfer_opts.inv_r (or folds 1/r into A).
 *
 * All arithmetic is fp64 (samples widened exactly).  Conventions as above:
 * device pointers are caller-owned HIP memory, nothing is allocated, scratch
 * comes from the workspace, work is enqueued on `stream` and no call
 * synchronizes the host.
 */

/*
 * Weighted sender RMS, means and joint covariance (Eq. 3; Sec. 3.2).
 *   n          samples, >= 1.
 *   p, q       feature sizes, each in [1, 65536].
 *   dtype      HF_F32 or HF_BF16: storage of x and y.
 *   x          device [n][ldx], row n holds x_n in its first p entries (ldx >= p).
 *   y          device [n][ldy], y_n in the first q entries (ldy >= q).
 *   w          device fp32 [n] sample weights (>= 0, positive sum), or NULL for 1.
 *   r          device fp64 [1]: r = sqrt(sum w |x|^2 / (p sum w)).
 *   mu         device fp64 [p + q]: weighted means of z = x / r, then of y.
 *   cov        device fp64 [(p + q)^2] row-major: the joint covariance of
 *              [z | y], normalized by sum w (blocks S_Z, S_ZY / S_YZ, S_Y).
 *              Exactly symmetric.
 *   workspace  device, >= hf_recolor_moments_workspace_bytes(n, p, q), 256-B aligned.
 * The covariance is accumulated over centred samples (two passes).  A weight
 * sum of zero gives NaN results.
 */
size_t hf_recolor_moments_workspace_bytes(int64_t n, int32_t p, int32_t q);
int32_t hf_recolor_moments(int64_t n, int32_t p, int32_t q, int32_t dtype, const void* x,
                           int64_t ldx, const void* y, int64_t ldy, const float* w, double* r,
                           double* mu, double* cov, void* workspace, size_t workspace_bytes,
                           void* stream);

/* Convergence of the three Newton-Schulz iterations of hf_recolor_solve
 * (index 0: roots of S_Z, 1: roots of S_Y, 2: the Procrustes factor). */
typedef struct {
  int32_t iterations[3];  /* steps taken */
  int32_t converged[3];   /* 1: residual below 1e-3 and three more steps taken */
  double residual[3];     /* last |I - P|_F (P = Z Y for the roots, X^T X or X X^T) */
} hf_recolor_info;

/*
 * Recolor initialization from moments (Eq. 4-5).
 *   p, q       as in hf_recolor_moments.
 *   mu, cov    device fp64: hf_recolor_moments' outputs (or any means and SPD
 *              joint covariance in that layout).
 *   ridge      >= 0: S + ridge * (trace S / dim) * I replaces S_Z and S_Y
 *              before their roots (the paper's numerical stabilization is
 *              unspecified; 0 is the unregularized map).
 *   A          device fp64 [q][p] (out).
 *   b          device fp64 [q] (out).
 *   info       device hf_recolor_info (out), or NULL.
 *   workspace  device, >= hf_recolor_solve_workspace_bytes(p, q), 256-B aligned.
 * Method: the symmetric roots S^{1/2}, S^{-1/2} by the coupled Newton-Schulz
 * iteration after scaling S by its Frobenius norm; R* as the polar factor of
 * the whitened cross-covariance by the Newton-Schulz polar iteration (equal to
 * U Q^T when that matrix has full rank).  Each iteration stops three steps
 * after its residual falls below 1e-3, or after 64 (roots) / 128 (polar)
 * steps; the call returns before the device finishes, so read info after the
 * stream completes: converged[i] == 0 means the result is not valid (a
 * singular covariance without ridge, or a rank-deficient cross-covariance).
 */
size_t hf_recolor_solve_workspace_bytes(int32_t p, int32_t q);
int32_t hf_recolor_solve(int32_t p, int32_t q, const double* mu, const double* cov, double ridge,
                         double* A, double* b, hf_recolor_info* info, void* workspace,
                         size_t workspace_bytes, void* stream);

/*
 * Fold a rank-`rank` correction y^ = y0 + (y0 B) G into the map (Eq. 9):
 * the paper's A (I + B G) and b (I + B G), in the stored orientation
 * A_out = A + G^T (B^T A), b_out = b + G^T (B^T b).
 *   A, b       device fp64 [q][p] and [q] (e.g. from hf_recolor_solve).
 *   B          device fp64 [q][rank] (the paper's B, d_R x rho).
 *   G          device fp64 [rank][q].
 *   A_out, b_out  device fp64 [q][p], [q]; may be A and b themselves.
 *   rank       >= 1.
 *   workspace  device, >= hf_fold_workspace_bytes(p, rank), 256-B aligned.
 */
size_t hf_fold_workspace_bytes(int32_t p, int32_t rank);
int32_t hf_fold_map(int32_t p, int32_t q, int32_t rank, const double* A, const double* b,
                    const double* B, const double* G, double* A_out, double* b_out,
                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * The fp64 matrix-core product behind the three calls above, exposed for
 * testing and reuse: D = alpha * op(A) op(B) + beta * C + gamma * I, where
 * op(A) is m x k, element (i, kk) at A[kk * lda + i] when a_kmajor else
 * A[i * lda + kk], and op(B) is k x n, element (kk, j) at B[kk * ldb + j] when
 * b_kmajor else B[j * ldb + kk].  D is [m][ldd] row-major; C (read only when
 * beta != 0) is [m][ldc] and may be D.  m, n >= 1, k >= 0.
 */
int32_t hf_gemm_f64(int32_t m, int32_t n, int64_t k, const double* A, int64_t lda,
                    int32_t a_kmajor, const double* B, int64_t ldb, int32_t b_kmajor, double* D,
                    int64_t ldd, double alpha, double beta, const double* C, int64_t ldc,
                    double gamma, void* stream);

/* ------------------------------------------------------------------------ */
/* Kernel timing (tracing).                                                  */
/* ------------------------------------------------------------------------ */

typedef enum {
  HF_KERNEL_TRANSFER = 0,   /* the main transfer kernel of hf_transfer_kv */
  HF_KERNEL_ROPE_TABLES = 1,/* cos/sin table kernel of hf_transfer_kv */
  HF_KERNEL_ALIGNMENT = 2,  /* the three kernels of hf_build_alignment, together */
  HF_KERNEL_PACK = 3,       /* hf_pack_maps */
  HF_KERNEL_MOMENTS_STATS = 4, /* hf_recolor_moments: column statistics, then the sum of
                                  the covariance partials (two timed groups per call) */
  HF_KERNEL_MOMENTS_COV = 5,   /* hf_recolor_moments: the covariance product kernel */
  HF_KERNEL_RECOLOR_SOLVE = 6, /* all launches of hf_recolor_solve */
  HF_KERNEL_FOLD = 7,          /* all launches of hf_fold_map */
  HF_KERNEL_TRANSFER_STAGE = 8,/* per-tile alignment staging of hf_transfer_kv (bf16, tiled) */
  HF_KERNEL_STAGED_BUILD = 9,  /* staged path: aligned features of every slab to the workspace */
  HF_KERNEL_STAGED_GEMM = 10,  /* staged path: the map products with bias and RoPE */
  HF_KERNEL_COUNT = 11
} hf_kernel_id;

/*
 * While enabled (on != 0), every launch of the kernels above is bracketed by
 * a pair of HIP events recorded on its own stream.  hf_profiler_query waits
 * for the recorded events and returns the summed duration in milliseconds and
 * the number of launches since the last reset.  Host-thread safe.
 */
int32_t hf_profiler_enable(int32_t on);
int32_t hf_profiler_reset(void);
int32_t hf_profiler_query(int32_t kernel_id, double* total_ms, int64_t* launches);
/*
 * Per-launch durations (ms) of one kernel since the last reset, oldest
 * first: the first min(capacity, count) of them are copied to ms (host,
 * caller-owned; the profiler keeps at most 4096 per kernel) and *count gets
 * how many it keeps.  Waits for the recorded events like hf_profiler_query.
 */
int32_t hf_profiler_samples(int32_t kernel_id, float* ms, int64_t capacity, int64_t* count);

#ifdef __cplusplus
}
#endif

#endif /* HETEROFOLD_H */
