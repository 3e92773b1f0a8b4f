/*
 * nystra.h -- C ABI of the MI355X (gfx950) PnP-Nystra window-attention library.
 *
 * PnP-Nystra ("Plug-and-Play Linear Attention with Provable Guarantees for
 * Training-Free Image Restoration") replaces softmax self-attention inside
 * window-based restoration Transformers by a Nystrom approximation of the
 * exponential kernel G = exp(Q K^T / sqrt(d)) (Eqs. (2)-(7)), computed in the
 * row-max-stabilised form of Eq. (8) (Sec. 2.2), independently for every
 * (window, head) pair -- a "unit".
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Tensors.  Q, K, V, O are caller-owned DEVICE buffers, contiguous as
 *   [n_windows][heads][N][d_h] with element type `dtype` (NYSTRA_F32 = IEEE
 *   binary32, NYSTRA_BF16 = bfloat16).  Tokens of a window are row-major over
 *   its sqrt(N) x sqrt(N) pixel grid (SwinIR / Uformer window partition); the
 *   value width equals d_h.  O has the input dtype; bf16 outputs are rounded
 *   to nearest-even from an fp32 result.
 * Arithmetic.  fp32 inputs: fp32 throughout (fp32 matrix cores, fp32 VALU).
 *   bf16 inputs: the stored bf16 values are exact operands; landmark means,
 *   logits, row maxima, exponentials, sums and the Step 7 division are fp32.
 *   The contractions of the MFMA-tiled and token-split kernels (S_L, S_U,
 *   T = G_U^n [V | 1], O = G_L^n W and the Step 4 products) run on the bf16
 *   matrix cores with fp32 accumulation, every fp32 operand carried as two
 *   bf16 terms hi = bf16(x), lo = bf16(x - hi) (about 16 significant bits).
 *   Where both factors are split, the 64-token kernel forms all four term
 *   products; the larger-window and token-split kernels drop lo x lo (a
 *   2^-16 relative term).  S_A and W = Z T stay fp32.  The resulting error
 *   is ~1e-4 of the output RMS, far below the bf16 rounding of O.  The exact
 *   kernel (nystra_exact_attn_forward) in bf16 rounds its probabilities to
 *   bf16 for the P V product, as bf16 flash attention does (row sums fp32).
 * Streams.  `stream` is a hipStream_t (NULL = the null stream).  Work is
 *   enqueued and the call returns at once; the library never synchronises,
 *   allocates no device memory and keeps no mutable global state (apart from
 *   the static scratch of nystra_attn_forward_noalloc), so calls on
 *   different streams may overlap.  Only kernel launches are enqueued (no
 *   memory fills or copies), so a call can be recorded in a HIP graph.
 *   Faults inside a kernel surface at the caller's next synchronisation.
 * Errors.  Every function returns an int status (nystra_status).  All
 *   argument checks run before anything is enqueued, so on any error other
 *   than NYSTRA_ERR_HIP no output is written.  n_windows == 0 or heads == 0
 *   is a valid no-op (pointers may then be NULL).  NYSTRA_ERR_HIP reports a
 *   failed launch; nystra_last_error() then holds the HIP message for the
 *   calling thread.  Each entry point clears the thread's pending HIP error
 *   (hipGetLastError) right before it launches, so an error left by an
 *   earlier, unrelated HIP call is not reported as its own.  Nothing throws
 *   or aborts across this boundary.
 * Limits.  1 <= N <= 2^20, 1 <= d_h <= 128, 1 <= m <= min(N, 64),
 *   n_windows * heads <= 2^24 - 1 (every grid stays under 2^32 work-items),
 *   0 <= pinv_iters <= 64.  Pointers must be aligned to the element size.
 *   O must not overlap Q, K or V (Q, K, V may alias each other).
 */
#ifndef NYSTRA_H
#define NYSTRA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { NYSTRA_F32 = 0, NYSTRA_BF16 = 1 } nystra_dtype;

/* Landmark selection, Step 1 of Algorithm 1: landmarks are the means of the
 * tokens in non-overlapping pooling windows (Sec. 2.2).
 *  NYSTRA_LM_POOL2D:    the sqrt(N) x sqrt(N) token window is cut into m equal
 *                       rectangular patches on a g_r x g_c grid, g_c being the
 *                       largest divisor of m with g_c^2 <= m such that g_c and
 *                       g_r = m / g_c both divide sqrt(N); landmarks numbered
 *                       row-major over the patch grid.  Square m gives plain
 *                       2-D average pooling.  Requires N to be a square.
 *  NYSTRA_LM_SEGMENT1D: m contiguous runs of N/m tokens (requires m | N). */
typedef enum { NYSTRA_LM_POOL2D = 0, NYSTRA_LM_SEGMENT1D = 1 } nystra_landmark_mode;

/* Kernel family.  AUTO picks, for nystra_attn_forward_ex, the MFMA-tiled
 * kernel when the shape is one it covers and the pointers are aligned as it
 * needs (for bf16, Q, K, V and O to 4 bytes; fp32 needs nothing beyond the
 * element size), and the generic kernel otherwise; nystra_attn_forward_ws may in addition pick the
 * token-split kernels (see there).  The other values force one
 * (NYSTRA_ERR_UNSUPPORTED if it cannot run this shape, or -- for SPLIT -- if
 * the entry point takes no workspace). */
typedef enum {
    NYSTRA_VARIANT_AUTO = 0,
    NYSTRA_VARIANT_GENERIC = 1,
    NYSTRA_VARIANT_TILED = 2,
    NYSTRA_VARIANT_SPLIT = 3
} nystra_variant;

typedef enum {
    NYSTRA_OK = 0,
    NYSTRA_ERR_NULL = 1,        /* a required pointer is NULL                  */
    NYSTRA_ERR_SHAPE = 2,       /* sizes out of range or no pooling grid       */
    NYSTRA_ERR_DTYPE = 3,       /* dtype not NYSTRA_F32 / NYSTRA_BF16          */
    NYSTRA_ERR_ALIGN = 4,       /* pointer not aligned to the element size     */
    NYSTRA_ERR_OVERLAP = 5,     /* O overlaps Q, K or V                        */
    NYSTRA_ERR_UNSUPPORTED = 6, /* forced variant cannot run this shape        */
    NYSTRA_ERR_HIP = 7,         /* kernel launch failed (see nystra_last_error) */
    NYSTRA_ERR_ARG = 8,         /* other bad argument (mode, iters, scale)     */
    NYSTRA_ERR_WORKSPACE = 9    /* workspace missing, too small or misaligned  */
} nystra_status;

typedef struct nystra_opts {
    int pinv_iters;    /* Step 4 iterations K, 0..64; default 6                */
    int landmark_mode; /* nystra_landmark_mode; default NYSTRA_LM_POOL2D       */
    float scale;       /* logit scale; <= 0 selects 1/sqrt(d_h) (default 0)     */
    int variant;       /* nystra_variant; default NYSTRA_VARIANT_AUTO           */
} nystra_opts;

/* Fill *opts with the defaults above.  Returns NYSTRA_ERR_NULL for NULL. */
int nystra_default_opts(nystra_opts *opts);

/* PnP-Nystra forward (Algorithm 1, stabilised form Eq. (8)) with default
 * options: K = 6 pseudo-inverse iterations, POOL2D landmarks, scale
 * 1/sqrt(d_h).  For every unit:
 *   Qbar, Kbar = pooled landmark queries / keys (m x d_h)            Step 1
 *   m_L(i) = max_j (s Q Kbar^T)_ij,   G_L^n = exp(s Q Kbar^T - m_L)  Step 3
 *   m_U(i) = max_j (s Qbar K^T)_ij,   G_U^n = exp(s Qbar K^T - m_U)  Step 3
 *   G_A^n = exp(s Qbar Kbar^T - m_U)  (rows scaled by m_U)            Step 2
 *   Z = K iterations of Z <- Z(13I - AZ(15I - AZ(7I - AZ)))/4 on
 *       A = G_A^n from Z_0 = A^T / (||A||_1 ||A||_inf)                Step 4
 *   O = (G_L^n Z G_U^n V) / (G_L^n Z G_U^n 1_N)  row-wise             Steps 5-7
 * The products of Steps 5-6 are evaluated as G_L^n (Z (G_U^n [V | 1])),
 * which equals the paper's (G_L^n Z)(G_U^n [V | 1]) in exact arithmetic.
 * No epsilon is added to the denominator (Step 7). */
int nystra_attn_forward(const void *Q, const void *K, const void *V, void *O,
                        int n_windows, int heads, int N, int d_h, int m, int dtype,
                        void *stream);

/* As nystra_attn_forward with explicit options (opts == NULL: defaults). */
int nystra_attn_forward_ex(const void *Q, const void *K, const void *V, void *O,
                           int n_windows, int heads, int N, int d_h, int m, int dtype,
                           const nystra_opts *opts, void *stream);

/* Token-split PnP-Nystra for windows with many tokens and few units (global
 * attention: one window per feature map, N up to 2^20).  The same
 * computation as nystra_attn_forward_ex (Algorithm 1, Eq. (8)), organised as
 * six launches on `stream` so that every pass has thousands of workgroups:
 * landmark pooling in patch pieces (Step 1); per key chunk the row maxima of
 * S_U over the chunk and G_U^n [V | 1] against them; the chunk results merged
 * against the global row maxima m_U (Step 3, G_U side -- the sums are those of
 * the one-pass form, only added in another order); the landmark core per unit
 * (Steps 2, 4, 5-6); and per query chunk Steps 3 (G_L side), 6 and 7.
 *
 * nystra_attn_workspace_size stores in *bytes the device workspace that
 * nystra_attn_forward_ws needs for these arguments: 0 unless the call would
 * run the token-split kernels.  AUTO chooses them when the shape is supported
 * (N % 16 == 0, d_h a multiple of 4 in 8..32 or 30, m <= 64; for bf16, Q, K, V 4-byte
 * aligned; O 16-byte aligned) and N >= 4096, or N >= 2048 with fewer than 512
 * units; NYSTRA_VARIANT_SPLIT forces them.  The size depends on the arguments
 * only, not on any pointer (aligned tensors are assumed), and is about
 * units x (N / chunk) x 8.7 KB for key chunks of 256..4096 tokens.  Host-only.
 *
 * nystra_attn_forward_ws: as nystra_attn_forward_ex, with `workspace` a
 * caller-owned DEVICE buffer of at least the size above, 256-byte aligned and
 * disjoint from Q, K, V and O (NYSTRA_ERR_WORKSPACE otherwise; it may be NULL
 * when the size is 0).  Its contents on entry do not matter and on return are
 * unspecified; calls that may run concurrently need distinct workspaces.
 * Nothing is allocated. */
int nystra_attn_workspace_size(int n_windows, int heads, int N, int d_h, int m, int dtype,
                               const nystra_opts *opts, size_t *bytes);

int nystra_attn_forward_ws(const void *Q, const void *K, const void *V, void *O,
                           int n_windows, int heads, int N, int d_h, int m, int dtype,
                           const nystra_opts *opts, void *workspace, size_t workspace_bytes,
                           void *stream);

/* For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc: the same
 * computation and kernel choice as nystra_attn_forward_ws (AUTO may pick the
 * token-split kernels), with the token-split workspace taken from a static
 * device array of NYSTRA_STATIC_SCRATCH_BYTES (32 MiB) that the library holds
 * on every device it runs on, until the process ends (enough for global
 * attention over a 1024 x 1024 map with 6 heads of 30).  Nothing is
 * allocated.  The array belongs to the current device; `stream` (NULL = the
 * null stream) must belong to that device too (NYSTRA_ERR_ARG otherwise).
 * A call whose token-split workspace would exceed the array returns
 * NYSTRA_ERR_WORKSPACE before anything is enqueued.  Every call on a device
 * shares its array, whose contents on entry do not matter and on return are
 * unspecified: calls that overlap on one device (other streams or threads)
 * race on it and must be serialised by the caller.  The first call on a
 * device looks the array's address up (hipGetSymbolAddress). */
#define NYSTRA_STATIC_SCRATCH_BYTES (32u << 20)

int nystra_attn_forward_noalloc(const void *Q, const void *K, const void *V, void *O,
                                int n_windows, int heads, int N, int d_h, int m, int dtype,
                                const nystra_opts *opts, void *stream);

/* Window-attention block around the operator: the structure of Sec. 1 for
 * SwinIR / Uformer-style models, from a feature map X to a feature map Y.
 *   1. the B x H x W map is rolled by -shift in both directions and cut into
 *      (H / window) x (W / window) windows of N = window^2 tokens (windows
 *      numbered image-major, then row-major; tokens row-major);
 *   2. Q, K, V = X_win W_qkv + b_qkv (W_qkv [C][3C]: Q, K, V column blocks,
 *      head j taking columns j d_h .. (j+1) d_h - 1 of each, d_h = C / heads);
 *   3. per (window, head): PnP-Nystra (as nystra_attn_forward_ws, with m and
 *      opts) or, with attention = NYSTRA_BLOCK_EXACT, exact softmax attention
 *      (opts->scale only);
 *   4. heads concatenated, Y_win = O W_proj + b_proj (W_proj [C][C]);
 *   5. every token written back to its pixel (the roll undone).
 * Relative-position bias and the shifted-window mask are not applied (they
 * are not part of Eqs. (1)-(8)).
 * X, Y: [batch][height][width][channels] DEVICE buffers in `dtype`; weights
 * and biases in `dtype` (biases may be NULL: zero).  Q, K, V and the
 * attention output are stored in `dtype` in the workspace (as a model in that
 * dtype stores them); products accumulate in fp32 on the matrix cores.
 * Limits: window divides height and width, 0 <= shift < window, heads
 * divides channels, d_h <= 128, channels <= 4096, batch * height * width
 * <= 2^31 - 1, and the attention limits above for N, m and the unit count.
 * nystra_block_workspace_size: host-only size of the workspace
 * nystra_block_forward needs (Q, K, V, O, for channels <= 256 the two weight
 * matrices repacked into the GEMM's tile layout (written by each call), and
 * for long windows the token-split workspace).  nystra_block_forward: workspace as for
 * nystra_attn_forward_ws (256-byte aligned, disjoint from every other
 * argument, NYSTRA_ERR_WORKSPACE otherwise); Y must not overlap X, the
 * weights or the biases. */
typedef struct nystra_block_shape {
    int batch, height, width, channels, heads, window, shift;
} nystra_block_shape;

typedef enum { NYSTRA_BLOCK_NYSTROM = 0, NYSTRA_BLOCK_EXACT = 1 } nystra_block_attention;

int nystra_block_workspace_size(const nystra_block_shape *shape, int m, int dtype,
                                const nystra_opts *opts, int attention, size_t *bytes);

int nystra_block_forward(const void *X, const void *Wqkv, const void *bqkv, const void *Wproj,
                         const void *bproj, void *Y, const nystra_block_shape *shape, int m,
                         int dtype, const nystra_opts *opts, int attention, void *workspace,
                         size_t workspace_bytes, void *stream);

/* The block with its projection weights packed once (inference, where W_qkv
 * and W_proj do not change between calls; the same Sec. 1 block as above).
 * nystra_block_packed_size: host-only bytes of the packed image of W_qkv and
 * W_proj for `channels` and `dtype` (0 for channels > 256, where the block
 * reads the weights as given).
 * nystra_block_pack_weights: enqueues on `stream` the packing of Wqkv
 * [C][3C] and Wproj [C][C] (device, `dtype`, element-aligned) into `packed`
 * (device, 256-byte aligned, at least that size, disjoint from the weights;
 * caller-owned).  A no-op for channels > 256.
 * nystra_block_forward_packed: nystra_block_forward with the packing step
 * skipped: the GEMMs read `packed`, which must hold the image of the same
 * Wqkv and Wproj for these channels and dtype (its contents are not checked;
 * repack after changing the weights).  `packed` is required (NYSTRA_ERR_NULL)
 * for channels <= 256, ignored above; `packed_bytes` at least
 * nystra_block_packed_size (NYSTRA_ERR_WORKSPACE), 256-byte aligned
 * (NYSTRA_ERR_ALIGN) and disjoint from Y and the workspace
 * (NYSTRA_ERR_OVERLAP).  Every other argument, the workspace size included,
 * is as for nystra_block_forward.
 * Results are identical to nystra_block_forward's. */
int nystra_block_packed_size(int channels, int dtype, size_t *bytes);

int nystra_block_pack_weights(const void *Wqkv, const void *Wproj, int channels, int dtype,
                              void *packed, size_t packed_bytes, void *stream);

int nystra_block_forward_packed(const void *X, const void *Wqkv, const void *bqkv,
                                const void *Wproj, const void *bproj, const void *packed,
                                size_t packed_bytes, void *Y, const nystra_block_shape *shape,
                                int m, int dtype, const nystra_opts *opts, int attention,
                                void *workspace, size_t workspace_bytes, void *stream);

/* Exact windowed softmax self-attention, Eq. (1), per unit:
 *   O = softmax(scale Q K^T) V, with the row maximum subtracted inside the
 *   softmax.  scale <= 0 selects 1/sqrt(d_h).  Same layout, limits and
 *   conventions as nystra_attn_forward (no m). */
int nystra_exact_attn_forward(const void *Q, const void *K, const void *V, void *O,
                              int n_windows, int heads, int N, int d_h, int dtype,
                              float scale, void *stream);

/* Step 1 alone (landmark pooling, Sec. 2.2).  Writes the fp32 landmark
 * queries and keys Qbar, Kbar, each [n_windows][heads][m][d_h], and, if
 * `map` is not NULL, the int32[N] token -> landmark map (device memory).
 * Qbar, Kbar must not overlap Q, K; they must be 4-byte aligned. */
int nystra_landmark_pool(const void *Q, const void *K, float *Qbar, float *Kbar,
                         int32_t *map, int n_windows, int heads, int N, int d_h, int m,
                         int dtype, int mode, void *stream);

/* Host-only: the token -> landmark map of Step 1 into map_host[N]. */
int nystra_landmark_map(int N, int m, int mode, int32_t *map_host);

/* Host-only: which kernel family nystra_attn_forward_ex would launch for
 * this shape and options with aligned tensors (NYSTRA_VARIANT_GENERIC
 * or NYSTRA_VARIANT_TILED), or a negative nystra_status if the arguments are
 * invalid (NYSTRA_VARIANT_SPLIT, which needs a workspace, gives
 * -NYSTRA_ERR_UNSUPPORTED). */
int nystra_select_variant(int N, int d_h, int m, int dtype, const nystra_opts *opts);

/* Static description of a status code. */
const char *nystra_status_str(int status);

/* Detail of the last NYSTRA_ERR_HIP on the calling thread ("" if none). */
const char *nystra_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* NYSTRA_H */
