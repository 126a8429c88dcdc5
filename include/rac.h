/*
 * rac.h - C ABI of the MI355X (gfx950) RAC aligned residual codec.
 *
 * The codec is the one of the paper's Section "Quality- and Cost-Constrained
 * Aligned Residual Encoding".  A boundary hidden state H ([tokens x hidden],
 * bf16, row-major) is coded against a reference R of the same shape:
 *
 *   1. grouped affine alignment (Eq. affine-fit): for every token row and
 *      every group of g_a channels, the least-squares pair (alpha*, beta*) of
 *      x ~ alpha*r + beta; a zero-variance reference group gives alpha* = 0,
 *      beta* = mean(x).  Both ends use the fp16-serialized pair.
 *   2. aligned residual (Eq. aligned-residual): E = H - (alpha R + beta).
 *   3. outliers (paragraph "Outlier Metadata and Calibration"): optionally the
 *      k largest |E| of each token row leave the dense base and travel as
 *      (channel, fp16 value); ties go to the lower channel.  With
 *      RAC_FLAG_GROUP_OUTLIERS the scope is the paragraph's own: the k_g
 *      largest |E| of every quantization group, sent as u8 in-group offsets
 *      and fp16 values.
 *   4. grouped symmetric quantization (Eq. residual-quantization): per group of
 *      g_q channels, Qmax = 2^(q-1)-1, the scale is the smallest fp16 s with
 *      s*Qmax >= max|E^d| (rounded up, so nothing clips), codes are
 *      round-half-even(E^d / s); an all-zero group carries scale 0.
 *   5. reconstruction (Eq. residual-reconstruction): H-hat = R~ + E-hat, with
 *      E-hat = q*s on the dense base and the fp16 value at outliers.
 *
 * Arithmetic is IEEE binary32 with a fixed evaluation order (pairwise sums
 * over channel order, two-pass centred moments, no contraction except the
 * aligned reference alpha*r + beta, which is rounded once), so the sender's
 * reconstruction, the receiver's decode and an independent CPU implementation
 * agree bit for bit.
 *
 * Conventions shared by every entry point:
 *   - All tensor and wire pointers are DEVICE pointers on the current HIP
 *     device; the caller owns every buffer.  The library allocates nothing,
 *     frees nothing, never synchronizes and keeps no global state.
 *   - bf16 tensors (x, ref) are passed as raw 16-bit patterns, row-major
 *     [tokens][hidden]; x, ref and xhat must be 16-byte aligned and the wire
 *     256-byte aligned.
 *   - Work is enqueued on `stream` (a hipStream_t; 0 is the null stream) and
 *     is stream-ordered; calls are reentrant.  Calls on different streams may
 *     run concurrently as long as their output buffers do not overlap.
 *   - Argument errors are reported synchronously, before anything is
 *     enqueued.  RAC_ERR_HIP reports a failed kernel launch.  Kernels never
 *     trap; inputs must be finite (results for NaN/Inf inputs are unspecified
 *     but every memory access stays in bounds).
 *   - Saturation is reported in the wire itself.  Coefficients, scales and
 *     outlier values are fp16 fields holding the IEEE result of their
 *     rounding: a value whose round-to-nearest-even overflows (|v| >= 65520)
 *     is stored as +-infinity, and the scale of a quantization group whose
 *     largest |E^d| exceeds 65504 * Qmax (no finite fp16 step covers it, so
 *     the no-clipping guarantee of Eq. residual-quantization fails and the
 *     codes clip) is +infinity.  Both ends compute with +-65504 wherever a
 *     field holds +-infinity, so the reconstruction stays finite.
 *     rac_saturation_summary reads a host copy of a wire for these marks.
 *
 * Wire format (little-endian, self-describing, all padding zero):
 *   header (256 B): u32 magic 'RAC1', u16 version 2, u16 flags (1 per-token
 *     outliers, 2 fixed step, 4 encoded against a zero reference, 8 per-group
 *     outliers, 16 coefficients pooled over segments), u32 tokens,
 *     u32 hidden, u32 g_a, u32 g_q, u8 bits, u8 coef fmt (1 = fp16 pair),
 *     u8 scale fmt (1 = fp16, 0 = absent), u8 outlier fmt (1 = u16 channel in
 *     the low half and fp16 value in the high half of a u32, 2 = per-group
 *     fp16 values and u8 offsets, 0 = absent), u16 k, u16 0, then u64 offsets
 *     of the coef, scale, code and outlier sections, the total size and the
 *     offset of the per-group offset array (0 without per-group outliers);
 *     sections start at 256-byte boundaries.
 *   coef   : fp16 [tokens][hidden/g_a][2]   (alpha, beta)
 *   scale  : fp16 [tokens][hidden/g_q]      (absent with RAC_FLAG_FIXED_STEP)
 *   codes  : u8   [tokens][hidden*bits/8]   channel c of a row occupies bits
 *            [c*bits, c*bits+bits) of the row's little-endian bit string, as
 *            bits-wide two's complement (INT4: two values per byte, even
 *            channel in the low nibble)
 *   outl   : u32  [tokens][k]               ascending channel per row
 *   per-group outliers instead (k = k_g):
 *   oval   : fp16 [tokens][hidden/g_q][k_g] at the outlier offset
 *   ooff   : u8   [tokens][hidden/g_q][k_g] in-group offsets, ascending within
 *            each group, aligned with oval
 *   every fp16 field may hold +-infinity, which stands for +-65504 and
 *   marks a saturation (see above)
 */
#ifndef RAC_H
#define RAC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* rac_stream_t; /* identical to hipStream_t */

typedef enum {
    RAC_OK = 0,
    RAC_ERR_INVALID = 1,     /* configuration or pointer argument invalid        */
    RAC_ERR_ALIGN = 2,       /* a pointer breaks the alignment rules above       */
    RAC_ERR_CAPACITY = 3,    /* wire buffer smaller than rac_wire_size()         */
    RAC_ERR_HIP = 4,         /* the HIP runtime refused the kernel launch        */
    RAC_ERR_FORMAT = 5,      /* a wire header does not parse                     */
    RAC_ERR_UNSUPPORTED = 6, /* valid codec configuration the kernels do not
                                implement (hidden above 8192; a gathered call
                                of more than 268,435,392 rows may be refused)   */
    RAC_ERR_NOMEM = 7        /* host memory exhausted (span index only)          */
} rac_status;

enum {
    /* Quantize with a calibrated step per channel group instead of the
     * per-(token, group) max-abs scale: s = smallest fp16 >= fixed_steps[g],
     * codes clip to +-Qmax, the wire carries no scale section. */
    RAC_FLAG_FIXED_STEP = 1u << 0,
    /* Write the reconstruction as bf16 (round to nearest even of the fp32
     * value) instead of fp32. */
    RAC_FLAG_XHAT_BF16 = 1u << 1,
    /* Outliers per quantization group (the outlier paragraph's mask M_j):
     * outlier_k is k_g, the number taken from every group of g_q channels
     * (ties to the lower channel), 1 <= k_g <= min(16, g_q/4), g_q <= 256. */
    RAC_FLAG_GROUP_OUTLIERS = 1u << 2,
    /* Launch hints; neither changes the wire or any result, only how rows are
     * spread over workgroups, and neither is recorded in the wire.  By default
     * more than 256 rows run on a grid of the workgroups the device holds at
     * once, each taking rows in strides with its next row prefetched, unless
     * that would give each more than six rows; then one workgroup per row
     * (over many rows the strided workgroups drift apart and the HBM writes
     * lose locality).  STRIDED always takes the strided grid, PER_ROW always
     * one workgroup per row; setting both is RAC_ERR_INVALID. */
    RAC_FLAG_LAUNCH_STRIDED = 1u << 3,
    RAC_FLAG_LAUNCH_PER_ROW = 1u << 4
};

typedef struct {
    int64_t tokens;      /* T = B*N token rows, 0 <= T < 2^31                      */
    int32_t hidden;      /* d: multiple of 8, 8 <= d <= 65535 (kernels: <= 8192)  */
    int32_t group_align; /* g_a: power of two, 8 <= g_a <= d, divides d           */
    int32_t group_quant; /* g_q: power of two, 8 <= g_q <= d, divides d           */
    int32_t bits;        /* q in {2, 3, 4, 8}; Qmax = 2^(q-1) - 1                  */
    int32_t outlier_k;   /* outliers per token row, 0 <= k <= min(64, d); with   */
                         /* RAC_FLAG_GROUP_OUTLIERS the k_g per group             */
    uint32_t flags;      /* RAC_FLAG_*                                            */
} rac_config;

typedef struct {
    uint64_t off_coef, off_scale, off_codes, off_outl, total; /* bytes */
    uint64_t off_ooff; /* per-group outlier offsets (0 without that mode) */
} rac_layout;

/* Host-only, pure.  Section offsets and total wire size for `cfg`.
 * Returns RAC_ERR_INVALID for a configuration outside the ranges above. */
rac_status rac_wire_layout(const rac_config* cfg, rac_layout* out);

/* Host-only, pure.  Total wire bytes for `cfg`, or 0 if it is invalid. */
size_t rac_wire_size(const rac_config* cfg);

/* Host-only, pure.  Parse a wire header the caller has copied to HOST memory
 * (at least 256 bytes) into `out` (flags gets RAC_FLAG_FIXED_STEP when the
 * wire carries no scales and RAC_FLAG_GROUP_OUTLIERS for per-group outliers).  Checks magic, version, field ranges and that the
 * recorded offsets match the layout of the parsed configuration; returns
 * RAC_ERR_FORMAT otherwise.  `zero_ref` (may be NULL) receives 1 when the
 * wire was encoded against a zero reference. */
rac_status rac_parse_header(const void* header_host, size_t len, rac_config* out,
                            int* zero_ref);

/* Host-only, pure.  Saturation marks of a wire produced for `cfg` that the
 * caller has copied to HOST memory (len >= rac_wire_size(cfg)): `rows` (may
 * be NULL) receives the number of token rows with any fp16 field holding
 * +-infinity, `bits` (may be NULL) the OR over the wire of 1 (an alpha or
 * beta), 2 (a scale; codes clipped) and 4 (an outlier value).  RAC_ERR_INVALID
 * for a bad configuration or a short buffer. */
rac_status rac_saturation_summary(const rac_config* cfg, const void* wire_host, size_t len, int64_t* rows,
                                  uint32_t* bits);

/* Sender side: encode x against ref into `wire`, and optionally write the
 * sender-side reconstruction H-hat into `xhat` in the same pass (the paper's
 * sender reconstruction, which keeps later references in sync with the
 * receiver).
 *   x           : bf16 [T][d]                          (required if T > 0)
 *   ref         : bf16 [T][d], or NULL for a zero reference
 *   fixed_steps : fp32 [d/g_q], only with RAC_FLAG_FIXED_STEP, else ignored
 *   wire        : u8 [wire_cap], wire_cap >= rac_wire_size(cfg); the first
 *                 rac_wire_size(cfg) bytes are written, header included
 *   xhat        : fp32 [T][d] (bf16 with RAC_FLAG_XHAT_BF16), or NULL
 * One kernel launch. */
rac_status rac_encode(const rac_config* cfg, const void* x, const void* ref,
                      const float* fixed_steps, void* wire, size_t wire_cap, void* xhat,
                      rac_stream_t stream);

/* Sender side: H-hat from a wire this sender produced (same definition and
 * same kernel as rac_decode, so the result is bit-identical to the fused
 * reconstruction of rac_encode and to the receiver's rac_decode).
 * Arguments as in rac_decode. */
rac_status rac_reconstruct(const rac_config* cfg, const void* wire, const void* ref,
                           const float* fixed_steps, void* xhat, rac_stream_t stream);

/* Receiver side (Eq. residual-reconstruction): H-hat = alpha*R + beta + E-hat
 * from the wire and the receiver's own reference.
 *   wire        : a wire produced for exactly `cfg` (device memory); the
 *                 header is not re-read on the device - a receiver that got
 *                 the wire from elsewhere checks it with rac_parse_header
 *   ref         : bf16 [T][d], or NULL for a zero reference
 *   fixed_steps : fp32 [d/g_q] with RAC_FLAG_FIXED_STEP, else ignored
 *   xhat        : fp32 [T][d] (bf16 with RAC_FLAG_XHAT_BF16)
 * Outlier entries whose channel is >= d (per-group entries: whose in-group
 * offset is >= g_q) are ignored.  One kernel launch. */
rac_status rac_decode(const rac_config* cfg, const void* wire, const void* ref,
                      const float* fixed_steps, void* xhat, rac_stream_t stream);

/* Encode against a gathered reference (the prefill uplink's retrieved spans):
 * the reference of token row t is row ref_rows[t] of `ref_store`, a
 * device-resident store of earlier reconstructions kept as bf16 (for example
 * the XHAT_BF16 output of earlier calls, which sender and receiver hold
 * bit-identical).  The reference rows are read from the store inside the
 * encode kernel, so the [T][d] reference is never materialized.  Everything
 * else is rac_encode: same wire, same reconstruction as rac_encode with a
 * reference whose row t is that store row.
 *   ref_store  : bf16 [store_rows][d], 16-byte aligned, or NULL for a zero
 *                reference on every row (then ref_rows is ignored)
 *   store_rows : 0 <= store_rows < 2^31
 *   ref_rows   : int32 [T] device array, 4-byte aligned, required with a
 *                store.  A negative index, or one >= store_rows, gives that
 *                token a zero reference row (no span hit); the kernels never
 *                read outside the store.
 * Errors as rac_encode, plus RAC_ERR_INVALID for a store without ref_rows or
 * store_rows out of range, and RAC_ERR_UNSUPPORTED for more token rows than
 * 64 per workgroup of the largest grid one dispatch holds (2^32 work-items);
 * that never happens for T <= 268,435,392.  One kernel launch. */
rac_status rac_encode_gather(const rac_config* cfg, const void* x, const void* ref_store, int64_t store_rows,
                             const int32_t* ref_rows, const float* fixed_steps, void* wire, size_t wire_cap,
                             void* xhat, rac_stream_t stream);

/* Receiver side of rac_encode_gather: rac_decode with the reference of token
 * row t taken from row ref_rows[t] of the receiver's own store (arguments as
 * in rac_encode_gather; the result equals rac_decode with that reference). */
rac_status rac_decode_gather(const rac_config* cfg, const void* wire, const void* ref_store, int64_t store_rows,
                             const int32_t* ref_rows, const float* fixed_steps, void* xhat, rac_stream_t stream);

/* Encode with the affine fit pooled over segments of rows: the affine-fit
 * equation over all fitting positions of a segment (for example one retrieved
 * span) instead of one row.  Segment s covers token rows
 * [seg_start[s], seg_start[s+1]); seg_start is a device int32 array of
 * segments + 1 entries with 0 = seg_start[0] < ... < seg_start[segments] = T
 * (bounds outside [0, T] are clamped on the device; other broken segmentations
 * give unspecified coefficients, never an access outside the buffers).  Per
 * (row, group) the centred moments are those of the per-token fit; the rows
 * of a segment are combined by the pairwise merge of centred moments over the
 * binary-decomposition tree (n rows split into the first p, p the largest
 * power of two below n, and the rest), so a one-row segment is exactly the
 * per-token fit.  Every row of a segment carries the segment's (alpha, beta),
 * the wire is otherwise the one of rac_encode (header flag 16 marks the
 * pooled fit) and rac_decode / rac_reconstruct read it unchanged.  Element
 * counts of a segment are exact in binary32 up to 2^24 (g_a * rows).
 * Requires g_a <= 512 and g_a * bits >= 128 (the row moments are staged in
 * the wire's code section before the codes overwrite them), else
 * RAC_ERR_UNSUPPORTED.  Three kernel launches on `stream`.  Other arguments
 * and errors as rac_encode. */
rac_status rac_encode_pooled(const rac_config* cfg, const void* x, const void* ref, int64_t segments,
                             const int32_t* seg_start, const float* fixed_steps, void* wire, size_t wire_cap,
                             void* xhat, rac_stream_t stream);

/* ---- Offline calibration -----------------------------------------------
 * The encoding subsection's opening paragraph, the last sentence of "Grouped
 * Residual Quantization" and "Outlier Metadata and Calibration": offline, the
 * sender's reconstruction path is run over candidate configurations (the
 * groupings g_a and g_q, the bit width q and, with outliers, the count k_g)
 * on a calibration sample, and a configuration meeting a quality target is
 * kept while the packed bytes (values, scales, coefficients, outliers) are
 * counted.  This library's reading: quality is the normalized squared error
 * NMSE = sum (x - H-hat)^2 / sum x^2 of the sender reconstruction; cost is
 * the configuration's whole wire (rac_wire_size); the choice is the fewest
 * bytes among candidates with NMSE <= target (ties: smaller squared error,
 * then the earlier candidate), or, when none meets the target, the smallest
 * squared error (ties: fewer bytes, then the earlier candidate). */

/* Host-only, pure.  Workspace bytes of rac_recon_error for `tokens` rows
 * (24 bytes per group of 8 rows), or 0 for a negative count. */
size_t rac_recon_error_workspace(int64_t tokens);

/* Reconstruction error of a coded sample: stats (a DEVICE double[3])
 * receives sum (x - H-hat)^2, sum x^2 and max |x - H-hat| in binary64 (each
 * difference and square one rounded binary64 operation, the sums in a fixed
 * order that does not depend on the device).
 *   x         : bf16 [tokens][hidden], 16-byte aligned
 *   xhat      : fp32 [tokens][hidden] (bf16 with RAC_FLAG_XHAT_BF16), 16-byte aligned
 *   flags     : 0 or RAC_FLAG_XHAT_BF16
 *   workspace : device scratch of rac_recon_error_workspace(tokens) bytes,
 *               8-byte aligned, owned by the caller (its contents on return
 *               are unspecified)
 * hidden must be a positive multiple of 8.  RAC_ERR_INVALID / RAC_ERR_ALIGN /
 * RAC_ERR_CAPACITY (workspace too small) are returned before any launch.  Two
 * kernel launches on `stream`. */
rac_status rac_recon_error(int64_t tokens, int32_t hidden, uint32_t flags, const void* x, const void* xhat,
                           double* stats, void* workspace, size_t workspace_bytes, rac_stream_t stream);

/* rac_recon_error for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same two kernel launches and the same result, bit for bit,
 * but the partials live in a fixed array inside the library (384 KiB per
 * device, held until the process ends) instead of a workspace.  This call
 * allocates nothing: on its first call on a device it looks up that array's
 * address (with the device current) and keeps it.  tokens is limited to
 * 131072 (RAC_ERR_CAPACITY beyond, before any launch).  Every call on one
 * device shares the array: calls that overlap on one device (different
 * streams, or different host threads) race and give unspecified results;
 * calls ordered on one stream are fine, and nothing left by an earlier call
 * is read.  Other arguments and errors as rac_recon_error. */
rac_status rac_recon_error_noalloc(int64_t tokens, int32_t hidden, uint32_t flags, const void* x, const void* xhat,
                                   double* stats, rac_stream_t stream);

/* One candidate of rac_calibrate: the configuration in, the measurements out. */
typedef struct {
    rac_config cfg;      /* in: tokens and hidden of the sample; no RAC_FLAG_FIXED_STEP */
    uint64_t wire_bytes; /* out: rac_wire_size(&cfg), the packed cost */
    double sq_err;       /* out: sum (x - H-hat)^2 over the sample */
    double sq_x;         /* out: sum x^2 */
    double max_abs;      /* out: max |x - H-hat| */
    double nmse;         /* out: sq_err / sq_x (0 when sq_x is 0) */
    int32_t feasible;    /* out: nmse <= target */
    int32_t reserved;
} rac_candidate;

/* Host-only, pure.  Workspace bytes rac_calibrate needs for these candidates
 * (a reconstruction of the sample, the largest wire, the error partials and
 * per-candidate sums), or 0 if a candidate is invalid, uses a step table,
 * exceeds the kernels' 8192 channels or differs from the first in tokens or
 * hidden. */
size_t rac_calibrate_workspace(const rac_candidate* candidates, int32_t n);

/* Offline calibration over n candidates (HOST array, filled in place) on the
 * sample x against ref (DEVICE bf16 [tokens][hidden]; ref NULL = zero
 * reference): for each candidate, rac_encode with the fused reconstruction,
 * then rac_recon_error of that reconstruction; then the choice above,
 * written to *chosen (a host int).  workspace: DEVICE memory of
 * rac_calibrate_workspace() bytes, 256-byte aligned.  Unlike every other
 * entry point, this offline routine reads its results back: it copies them
 * to the host and synchronizes `stream` before returning.  Argument errors
 * come before any launch; RAC_ERR_HIP if a launch, copy or the
 * synchronization fails. */
rac_status rac_calibrate(const void* x, const void* ref, rac_candidate* candidates, int32_t n, double target_nmse,
                         void* workspace, size_t workspace_bytes, int32_t* chosen, rac_stream_t stream);

/* ---- Decode-phase reference predictor ----------------------------------
 * Subsection "Predicted References for Decode", Eq. decode-predictor: from
 * the second decode step on, each boundary has a one-layer causal Transformer
 * that keeps a bounded causal state (a key-value cache) and maps the previous
 * reconstructed state H-hat^{t-1} of a sequence to the reference R_pred^t of
 * the current one.  The paper gives neither its sizes nor its trained
 * weights; this library's reading (the layers below) is a pre-norm block of
 * width `model` with `heads` heads of 64 channels and a SwiGLU of width
 * `ffn`, attending to the latest `window` inputs of the sequence with rotary
 * positions, between a projection from and a residual projection back to the
 * boundary width:
 *   h0 = x W_in^T                         x = H-hat^{t-1} (bf16 [B][hidden])
 *   q, k, v = RMSNorm(h0; g1) W_qkv^T     rotary: channel pair (2i, 2i+1) of
 *                                         each head turned by pos * 10000^(-2i/64)
 *   o  = softmax(q k^T / 8) v             over positions max(0, pos-window+1)..pos
 *   h1 = h0 + o W_o^T
 *   h2 = h1 + (silu(n2 W_gate^T) * (n2 W_up^T)) W_down^T,   n2 = RMSNorm(h1; g2)
 *   R  = x + RMSNorm(h2; g3) W_out^T      (bf16 [B][hidden])
 * RMSNorm(h; g) = h / sqrt(mean(h^2) + 1e-6) * g.  Products are bf16 x bf16
 * with fp32 accumulation; h0, h1, h2, q, k, v are fp32; the normalized
 * activations, o, the SwiGLU output, the cached keys (after rotation) and
 * values, and R are bf16 (round to nearest even). */
typedef struct {
    int32_t hidden;    /* boundary width d: multiple of 512, 512..8192           */
    int32_t model;     /* m: multiple of 128, 128..2048, = heads * 64            */
    int32_t heads;
    int32_t ffn;       /* SwiGLU width: multiple of 128, 128..8192               */
    int32_t window;    /* inputs attended (the bounded history): 1..1024         */
    int32_t max_batch; /* sequences per step: 1..256                             */
} rac_predictor_config;

/* Byte offsets of the weight blob's sections (bf16, each 256-byte aligned, in
 * this order): W_in [m][d], g1 [m], W_qkv [3m][m] (rows: the q, k, v outputs),
 * W_o [m][m], g2 [m], W_gu [2 ffn][m] (row 2j: gate j, row 2j+1: up j),
 * W_down [m][ffn], g3 [m], W_out [d][m]; every matrix is [outputs][inputs]. */
typedef struct {
    uint64_t w_in, g1, w_qkv, w_o, g2, w_gu, w_down, g3, w_out, total;
} rac_predictor_offsets;

/* Host-only, pure.  Weight blob layout; RAC_ERR_INVALID outside the ranges. */
rac_status rac_predictor_layout(const rac_predictor_config* cfg, rac_predictor_offsets* out);

/* Host-only, pure.  Bytes of the key-value cache: [max_batch][window][2][m]
 * bf16 (key, then value, of every position slot), or 0 for a bad config. */
size_t rac_predictor_cache_bytes(const rac_predictor_config* cfg);

/* Host-only, pure.  Bytes of the step's device scratch, or 0. */
size_t rac_predictor_workspace_bytes(const rac_predictor_config* cfg);

/* One decode step of `batch` sequences (batch <= max_batch).
 *   weights   : DEVICE blob (rac_predictor_layout), 256-byte aligned
 *   cache     : DEVICE [max_batch][window][2][model] bf16, caller-owned;
 *               sequence b's input at position p goes to slot p mod window;
 *               only slots of positions p - window + 1 .. p - 1 are read, so
 *               the cache needs no clearing and a restarted sequence (p = 0)
 *               reads nothing stale
 *   pos       : DEVICE int32 [batch], the input's 0-based position in its
 *               sequence (negative counts as 0)
 *   h_prev    : DEVICE bf16 [batch][hidden], the previous reconstructions
 *   ref_out   : DEVICE bf16 [batch][hidden], the predicted references
 *   workspace : DEVICE scratch of rac_predictor_workspace_bytes(), 256-byte aligned
 * Argument errors are returned before any launch.  Ten kernel launches on
 * `stream`. */
rac_status rac_predictor_step(const rac_predictor_config* cfg, const void* weights, void* cache, const int32_t* pos,
                              int32_t batch, const void* h_prev, void* ref_out, void* workspace,
                              size_t workspace_bytes, rac_stream_t stream);

/* ---- Reference selection for the prefill uplink (host only) ------------
 * Subsection "Repeated-Span Retrieval for Prefill Uplinks",
 * Eq. prefill-reference-selection.  A span index holds the token streams of
 * earlier requests and the store row of each of their tokens' activations;
 * rac_span_select turns the current prompt into the ref_rows array of
 * rac_encode_gather / rac_decode_gather.  Both ends can run it, since it
 * depends only on tokens.
 *
 * The index is a host object with an explicit lifetime (the one exception to
 * "the library allocates nothing": it holds host memory only, never device
 * memory).  Calls on one index must not overlap with rac_span_index_add on
 * the same index; concurrent rac_span_select calls are fine.
 *
 * Rule (every part of it is the paper's, the grouping of hash buckets by
 * window content is this library's reading):
 *   - every `window`-token window of the added requests is indexed; each
 *     distinct window content keeps its eight most recent occurrences
 *     (recency = request order, then position);
 *   - at prompt position i, each kept occurrence of the window starting at i
 *     extends forward to its longest exact match L >= window; the
 *     lexicographic maximum of (L, recency) is chosen and the scan moves to
 *     i + L (to i + 1 without a candidate);
 *   - the chosen span's positions i + o reference store row
 *     store_row0(request) + start + o; uncovered positions get -1 (no
 *     reference: rac_encode_gather codes them against zero). */
typedef struct rac_span_index rac_span_index;

/* New empty index over `window`-token windows, 1 <= window <= 4096.  NULL for
 * an invalid window or when host memory is exhausted. */
rac_span_index* rac_span_index_create(int32_t window);

/* Free an index (NULL is ignored). */
void rac_span_index_destroy(rac_span_index* index);

/* Add a request: host tokens[n]; the activation of token p is store row
 * store_row0 + p (store_row0 + n <= 2^31 - 1).  RAC_ERR_INVALID for bad
 * arguments, RAC_ERR_NOMEM if host memory runs out (the index may then hold
 * part of the request). */
rac_status rac_span_index_add(rac_span_index* index, const int32_t* tokens, int64_t n, int64_t store_row0);

/* Select the reference rows of a prompt: host tokens[n] -> host ref_rows[n]
 * (store row or -1).  `covered` (may be NULL) receives the number of
 * positions with a reference. */
rac_status rac_span_select(const rac_span_index* index, const int32_t* tokens, int64_t n, int32_t* ref_rows,
                           int64_t* covered);

/* Static string naming a status code. */
const char* rac_status_string(rac_status s);

#ifdef __cplusplus
}
#endif
#endif /* RAC_H */
