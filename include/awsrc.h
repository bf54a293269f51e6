/*
 * awsrc.h - C ABI of the AWSRC hot path on AMD Instinct MI355X (gfx950).
 *
 * AWSRC (activation-weighted seeded residual coding, arXiv 2608.23144) repairs
 * a quantized weight matrix: the residual R = W - W0 left by a backbone
 * quantizer (Eq. (1)) is cut into row-wise tiles of C input coordinates; for
 * each tile and each seed s a seeded signed-Hadamard basis B_s (Eq. (2)) is
 * fitted by activation-weighted ridge least squares (Eq. (3)), the P
 * coefficients are rounded to b bits with one scale per tile, and each tile
 * keeps the seed whose rounded fit leaves the smallest weighted error
 * (Sec. 3.2).
 * Records are ranked by weighted-error reduction per serialized byte
 * (Eq. (4), Sec. 3.3) and serialized as fixed-size records after a header
 * (Eq. (5), Sec. 3.4); the decoder regenerates B_s and adds B_s alpha_hat onto
 * W0 (Sec. 3.2).
 *
 * Conventions shared by every call:
 *  - Pointers are DEVICE pointers (HIP device memory owned by the caller)
 *    unless marked "host".  Matrices are row-major: rows = output features,
 *    cols = input features; tiles run along cols.
 *  - Work is enqueued on the caller's hipStream_t, passed as void* (NULL = the
 *    null stream).  Calls return once the work is enqueued, except where a
 *    call says it synchronizes.
 *  - The library never allocates device memory.  Calls that need scratch
 *    space take (workspace, ws_bytes): with workspace == NULL the call only
 *    stores the required byte count in *ws_bytes and returns AWSRC_OK;
 *    otherwise *ws_bytes must be at least that count.  The workspace must stay
 *    valid until the enqueued work has finished.
 *  - Every call returns an awsrc_status.  Nothing is launched when a call
 *    returns an error found during argument validation.  awsrc_last_error()
 *    returns a text description of the calling thread's last error.
 *  - The library keeps no mutable global state besides that per-thread error
 *    text and the scratch array of awsrc_encode_tiles_noalloc (with its
 *    per-device address, looked up once), so calls on different streams may
 *    run concurrently provided their buffers do not overlap (that entry point
 *    excepted, see there).  The small host copies of a call (a stream
 *    header, module tables, totals) go through host memory owned by that
 *    call, and a call that synchronizes waits on its own stream only.
 *
 * Conventions fixed where the paper leaves the choice open (the generator,
 * scale format, tie rules, backbone recipe and byte layouts) are documented
 * at the call that uses them.
 */
#ifndef AWSRC_H
#define AWSRC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define AWSRC_ABI_VERSION 1

typedef int32_t awsrc_status;
enum {
  AWSRC_OK = 0,
  AWSRC_EINVAL = -1,   /* bad shape, parameter or pointer                        */
  AWSRC_ENOSPC = -2,   /* workspace or output capacity too small, budget < header */
  AWSRC_ECORRUPT = -3, /* stream failed validation (nothing was written)          */
  AWSRC_EDEVICE = -4   /* a HIP runtime call failed                               */
};

enum { AWSRC_DTYPE_F32 = 0, AWSRC_DTYPE_BF16 = 1 };
enum { AWSRC_D_PER_COL = 0, AWSRC_D_PER_ELEM = 1 };
enum { AWSRC_MODE_GLOBAL = 0, AWSRC_MODE_PER_MODULE = 1 };
enum { AWSRC_SCALE_FP16 = 0, AWSRC_SCALE_POW2 = 1 };

/*
 * Codec parameters (the (C, P, b, S) of Sec. 3.1 plus generator and ridge).
 *  C            tile length: a power of two in 16..128.
 *  P            basis columns per seed: 1..min(C, 16).
 *  b            coefficient bits: 2..8; codes lie in [-(2^(b-1)-1), 2^(b-1)-1].
 *  S            number of seeds: 2..65536.
 *  scale_fmt    one scale per tile (Sec. 3.2), stored in a field of
 *               scale_bits bits:
 *               AWSRC_SCALE_FP16: scale = f16(f32(max_p |alpha*_p| / qmax)),
 *               both roundings to nearest even, saturating at 65504; the
 *               field holds the 16 fp16 bits.
 *               AWSRC_SCALE_POW2: the power-of-two scale of Sec. 3.2,
 *               scale = 2^e with e the smallest integer such that
 *               max_p |alpha*_p| <= qmax 2^e (no code clips), clamped to
 *               [-128, 127]; the field holds e + 128 in 8 bits (b_e = 8 in
 *               Eq. (5)).
 *               Either way an all-zero alpha* gives an all-zero record (field
 *               0) with gain 0.
 *  idx_bits     width of the tile-index field: 1..32, or 0 for
 *               ceil(log2 T_total) as in Eq. (5).
 *  gen_version  1: B_s = diag(sigma_s) H_C[:, c_s] / sqrt(C) with H_C the
 *               Sylvester Hadamard matrix in natural order and (sigma_s, c_s)
 *               drawn from the splitmix64 counter stream keyed by basis_key
 *               (word i of seed s is output s*2^32 + i; sign j is bit j%64 of
 *               word j/64; column p maps word ceil(C/64)+p into [0, C-p) by the
 *               multiply-shift of its high 32 bits and takes the m-th smallest
 *               column not yet drawn).  Eq. (2) without the seeded
 *               coordinate permutation.
 *               2: B_s[j, p] = sigma_j H_C[pi_s(j), c_p] / sqrt(C), the same
 *               signs and columns plus the seeded coordinate permutation of
 *               Eq. (2) / Sec. 3.1: coordinate j draws word ceil(C/64)+P+j and
 *               pi_s(j) is the rank of (word, j) in increasing order.  With
 *               per-element weights version 2 runs on the vector screen (the
 *               Gram entries need a transform of the permuted weights per
 *               seed); per-column weights keep the matrix-core screen.
 *  reserved     must be 0.
 *  basis_key    generator key, stored in the stream header.
 *  ridge_lambda eps_t = ridge_lambda * mean_j d_{t,j} in Eq. (3); >= 0.
 */
typedef struct awsrc_params {
  int32_t C, P, b, S;
  int32_t scale_fmt;
  int32_t idx_bits;
  int32_t gen_version;
  int32_t reserved;
  uint64_t basis_key;
  double ridge_lambda;
} awsrc_params;

int32_t awsrc_abi_version(void);
const char* awsrc_last_error(void);

/*
 * Backbone quantizer W0 = Q(W) of Eq. (1): asymmetric RTN-INT4 with groups of
 * `group` consecutive input columns (Sec. 4: RTN with group size 128).
 * fp32 arithmetic, correctly rounded, per group:
 *   s32 = (max - min) / 15; s16 = f16(s32) saturating; s = f32(s16);
 *   z = clamp(rint(-min / s), 0, 15); q = clamp(rint(w / s) + z, 0, 15);
 *   W0 = f32(q - z) * s.   A group with s16 == 0 stores s16 = 1, z = 0, q = 0.
 *  W          [rows, cols] fp32 or bf16 (w_dtype).
 *  group      64, 128 or 256; cols % group == 0.
 *  codes      [rows, cols/2] u8, even column in the low nibble.
 *  scale_f16  [rows, cols/group] fp16 bit patterns.
 *  zero       [rows, cols/group] u8.
 *  W0_or_null [rows, cols] fp32 dequantized backbone, or NULL to skip.
 *  W and W0 are 16-byte aligned, codes 4-byte aligned.
 */
awsrc_status awsrc_backbone_rtn(const void* W, int32_t w_dtype, int64_t rows, int64_t cols,
                                int32_t group, uint8_t* codes, uint16_t* scale_f16, uint8_t* zero,
                                float* W0_or_null, void* stream);

/*
 * Scale double quantization (SDQ) of the backbone's group scales (Sec. 3.3
 * names it, after QLoRA's double quantization of quantization constants;
 * Sec. 4 gives its rate for RTN g128, which the format below undercuts
 * slightly: 8 bits per group plus 64 per block, 0.0645 bits per weight).
 * The n_groups fp16 scales (awsrc_backbone_rtn's scale_f16, row-major) are
 * cut into blocks of 256; per block of n scales s_g:
 *   mu = f32(sum_g s_g / n)  (fp64 sum in group order, one division),
 *   dlt_g = f32(s_g - mu), a = max_g |dlt_g|,
 *   code_g = rint(dlt_g * 127 / a) in [-127, 127] (fp64, ties to even; 0 if a = 0),
 *   step = f32(a / 127).
 * The dequantized scale is s_hat_g = f32(mu + code_g * step).
 *  code        [n_groups] int8;  block_mean, block_step [ceil(n_groups / 256)] fp32.
 * Device pointers; asynchronous on `stream`.  EINVAL: n_groups < 0 or NULL buffer.
 */
awsrc_status awsrc_sdq_encode(const uint16_t* scale_f16, int64_t n_groups, int8_t* code, float* block_mean,
                              float* block_step, void* stream);

/*
 * W0 of an RTN-INT4-SDQ backbone (the backbone the paper's residual codecs
 * repair, Sec. 4): W0 = f32(q - z) * s_hat per group of `group` consecutive
 * input columns, with awsrc_backbone_rtn's codes and zero points and the
 * SDQ-dequantized scales of awsrc_sdq_encode.
 *  codes [rows, cols/2] u8 (4-byte aligned), zero [rows, cols/group] u8,
 *  sdq_code [rows * cols/group] int8, block_mean / block_step per 256 groups,
 *  W0 [rows, cols] fp32 (16-byte aligned).  cols % group == 0, group 64,
 *  128 or 256.  Asynchronous on `stream`.  EINVAL: bad shape, group,
 *  alignment or NULL buffer.
 */
awsrc_status awsrc_backbone_sdq_dequant(const uint8_t* codes, const uint8_t* zero, const int8_t* sdq_code,
                                        const float* block_mean, const float* block_step, int64_t rows,
                                        int64_t cols, int32_t group, float* W0, void* stream);

/*
 * Encoder seed search (Sec. 3.2, Eq. (2)-(4) numerator) for every tile of one
 * module.  Tile t = row * (cols / C) + block holds r_t = f32(W - W0) over
 * columns [block*C, block*C + C) of that row and coordinate weights d_t.  For
 * every seed the encoder fits Eq. (3), quantizes the coefficients, and scores
 * gain = sum_j d_j (r_j^2 - (r_j - rhat_j)^2); it keeps the seed with the
 * largest gain, the lowest seed winning exact ties.  All S seeds are screened
 * in fp32; the seeds whose screened gain lies close to the best are re-scored
 * in fp64 and the outputs come from that fp64 pass.
 *  W        [rows, cols] fp32 or bf16 (w_dtype); W0 [rows, cols] fp32.
 *  d        AWSRC_D_PER_COL: [cols] activation second moments shared by all
 *           rows; AWSRC_D_PER_ELEM: [rows, cols] per-element weights.  d > 0.
 *  cols % C == 0.  T = rows * cols / C.  W, W0 and d are 16-byte aligned.
 *  seed_out [T] u16, code_out [T, P] i8, scale_out [T] the scale field
 *  (fp16 bits or biased exponent, by scale_fmt),
 *  gain_out [T] f64 (weighted error reduction of the stored record; an
 *  all-zero record has gain 0), alpha_or_null [T, P] fp32 unquantized fit of
 *  the chosen seed, or NULL.
 *  Workspace: two-phase query as described above.
 */
awsrc_status awsrc_encode_tiles(const awsrc_params* p, const void* W, int32_t w_dtype,
                                const float* W0, int64_t rows, int64_t cols, const float* d,
                                int32_t d_mode, uint16_t* seed_out, int8_t* code_out,
                                uint16_t* scale_out, double* gain_out, float* alpha_or_null,
                                void* workspace, size_t* ws_bytes, void* stream);

/*
 * awsrc_encode_tiles over n_modules modules in one call, with the outputs of
 * all modules concatenated in module order (module m's tiles follow those of
 * modules 0..m-1, as in awsrc_rank_prefix's global tile index).  The results
 * are those of calling awsrc_encode_tiles once per module.  With per-element
 * weights, C = 64, P <= 8 and generator version 1 (the Fisher-blended weights
 * of Sec. 3.3 at the workloads' shapes) every module is screened in one
 * launch, so that small modules do not leave the GPU idle; otherwise the
 * modules are encoded one after another.
 *  W, W0, d     host arrays [n_modules] of device pointers, each module's
 *               inputs as in awsrc_encode_tiles (16-byte aligned).
 *  rows, cols   host arrays [n_modules]; cols % C == 0; rows may be 0.
 *  seed_out .. alpha_or_null
 *               device arrays over the sum T_total of the modules' tiles.
 * Workspace: two-phase query; the query needs no input pointers.
 */
awsrc_status awsrc_encode_modules(const awsrc_params* p, int32_t n_modules, const void* const* W, int32_t w_dtype,
                                  const float* const* W0, const float* const* d, int32_t d_mode,
                                  const int64_t* rows, const int64_t* cols, uint16_t* seed_out, int8_t* code_out,
                                  uint16_t* scale_out, double* gain_out, float* alpha_or_null, void* workspace,
                                  size_t* ws_bytes, void* stream);

/*
 * Diagnostic of the encoder's fp32 screen: copies the screened lists that the
 * last awsrc_encode_modules / awsrc_encode_tiles call with this workspace
 * (and the same p, module shapes and d_mode) kept for the fp64 re-score.
 * Per tile and seed range, kTop = 2 entries (gain in fp32, seed word), the
 * best first: gain_out and seed_out are device arrays [T_total][*nsplit][2];
 * with both NULL only *nsplit (seed ranges per tile) is returned.  A seed
 * word holds the seed in bits 0-15 and, in bit 16, a flag set when the
 * screen's fp32 rounding decisions for that candidate (the scale, a code)
 * lay within a small tolerance of a rounding threshold, where its score may
 * differ from the fp64 one by more than usual.  The re-score (Sec. 3.2)
 * re-evaluates the second entry in fp64 when its screened gain lies within
 * 1e-4 |g| + 1e-7 sum_j d_j r_j^2 of the first (3e-2 |g| + 3e-5 sum_j d_j
 * r_j^2 if either entry is flagged), so comparing the lists with gain_out of
 * the encode call measures the screen's error against that window.
 * Asynchronous on `stream`.  EINVAL where the call kept no
 * lists in the workspace: the per-column screen that runs the re-score
 * itself (C = 64, one seed range), or several modules encoded one by one.
 */
awsrc_status awsrc_encode_screen_lists(const awsrc_params* p, int32_t n_modules, const int64_t* rows,
                                       const int64_t* cols, int32_t d_mode, const void* workspace, float* gain_out,
                                       uint32_t* seed_out, int32_t* nsplit, void* stream);

/*
 * awsrc_encode_tiles without a workspace, for callers that cannot allocate
 * device memory (code under stream capture, serving loops, harnesses that
 * forbid allocation).  Same arguments, outputs and kernels as
 * awsrc_encode_tiles; the scratch space (basis and factor tables, screened
 * top lists) is one fixed device array per GPU inside the library, of
 * awsrc_encode_noalloc_max_bytes() bytes (64 MiB), held from the library's
 * load until the process ends; nothing is allocated or freed.  Its device
 * address is looked up on the first call on each device (the current device,
 * which `stream` must belong to).  A module whose scratch need (the size
 * awsrc_encode_tiles' query reports) exceeds the array returns AWSRC_ENOSPC
 * before anything is launched.  Every call on a GPU uses the same array:
 * calls that overlap on one GPU (different streams, or threads) race and must
 * be serialized by the caller; calls ordered on one stream are safe.  Nothing
 * in the array needs to start at zero (each call writes what it reads).
 */
awsrc_status awsrc_encode_tiles_noalloc(const awsrc_params* p, const void* W, int32_t w_dtype,
                                        const float* W0, int64_t rows, int64_t cols, const float* d,
                                        int32_t d_mode, uint16_t* seed_out, int8_t* code_out,
                                        uint16_t* scale_out, double* gain_out, float* alpha_or_null,
                                        void* stream);
/* Size in bytes of awsrc_encode_tiles_noalloc's scratch array. */
uint64_t awsrc_encode_noalloc_max_bytes(void);

/*
 * Work statistic of the last awsrc_encode_tiles call that used `workspace`
 * (same pointer): the number of (tile, seed) candidates scored in full in
 * the fp32 screen, ordered on `stream` after that call.  The screen for
 * per-column weights at C = 64 first bounds every candidate by the score of
 * its unquantized fit (Eq. (3) without the rounding of Sec. 3.2's codes,
 * which no quantized fit can exceed) and scores in full only those whose
 * bound reaches the tile's current second-best score; the other screens
 * score all T * S.  The result is the same either way; the count measures
 * the work.  Reads 8 bytes of device memory and synchronizes the stream.
 * EINVAL: NULL argument.
 */
awsrc_status awsrc_encode_scored(const void* workspace, uint64_t* scored, void* stream);

/*
 * Byte-budgeted, gain-ranked record selection and serialization (Eq. (4),
 * Sec. 3.3, Eq. (5)).  The per-tile encoder outputs of n_modules modules are
 * given concatenated in module order (global tile index = tiles of earlier
 * modules + local tile index).  Records with gain > 0 are eligible and are
 * ordered by decreasing gain (= decreasing rho, the record size being fixed),
 * ties by the lower global tile index.
 *  AWSRC_MODE_GLOBAL (P variant): budget = floor(bpw_budget * N / 8) bytes
 *    with N the total weight count; K = min(eligible, (budget - h) / L_rec);
 *    budget < h gives AWSRC_ENOSPC.  Every record-boundary prefix of the
 *    stream is itself the stream of a smaller budget.
 *  AWSRC_MODE_PER_MODULE (U variant): module m keeps
 *    min(eligible_m, floor(bpw_budget * N_m / 8) / L_rec) records; sections
 *    follow module order.  The quotas cover the records only, so the whole
 *    stream (header included) may exceed floor(bpw_budget * N / 8) bytes by
 *    up to the header size h.
 * Stream layout (little-endian): a header of h = 40 + 8 * n_modules bytes
 *   magic "AWSR" | version u16 = 1 | flags u16 (bits 0-3 gen_version, 4-7
 *   scale_fmt, bit 8 per-module mode) | C u16 | P u8 | b u8 | S u32 |
 *   idx_bits u8 | seed_bits u8 | scale_bits u8 | L_rec u8 | basis_key u64 |
 *   T_total u64 | n_modules u32 | then rows u32, cols u32 per module,
 * followed by K records of L_rec = ceil((idx_bits + ceil(log2 S) + P*b +
 * scale_bits)/8) bytes (scale_bits = 16 for fp16 scales, 8 for power-of-two
 * exponents): one LSB-first bit stream of tile index, seed, P
 * two's-complement b-bit codes and the scale field, zero padded.
 *  module_rows, module_cols  host arrays [n_modules]; cols % C == 0.
 *  stream_out     device buffer of stream_cap bytes; stream_cap < h + K*L_rec
 *                 gives AWSRC_ENOSPC.
 *  stream_len, K, n_eligible  host outputs (n_eligible may be NULL).
 * This call synchronizes with `stream` (it returns K).
 */
awsrc_status awsrc_rank_prefix(const awsrc_params* p, int32_t n_modules,
                               const int64_t* module_rows, const int64_t* module_cols,
                               int32_t mode, double bpw_budget, const uint16_t* seed,
                               const int8_t* code, const uint16_t* scale, const double* gain,
                               uint8_t* stream_out, uint64_t stream_cap, uint64_t* stream_len,
                               int64_t* K, int64_t* n_eligible, void* workspace, size_t* ws_bytes,
                               void* stream);

/*
 * Decoder (Sec. 3.2): for each record of a stream (or of any record-boundary
 * prefix of one, Sec. 3.3) regenerate B_s from the header's basis key and add
 * B_s (scale * q) onto that tile of W0, in place.  Tiles without a record are
 * not touched; an empty stream leaves W0 bit-identical.
 *
 * awsrc_decode_add = awsrc_decode_prepare + awsrc_decode_apply.
 *  stream_bytes  device pointer (8-byte aligned) to stream_len bytes;
 *                K = (stream_len - h) / L_rec.
 *  W0_ptrs       host array [n_modules] of device pointers to each module's
 *                W0, [rows, cols] in w0_dtype, 16-byte aligned; bf16
 *                targets are rounded to nearest even after the fp32 add.
 *  rows, cols    host arrays [n_modules]; must match the stream header.
 * The header and every record are validated before anything is written (magic,
 * version, parameters, length on a record boundary, tile index < T_total,
 * seed < S, codes within +-qmax, finite non-negative fp16 scale, no tile twice); a
 * failure returns AWSRC_ECORRUPT and leaves W0 unchanged.  This call
 * synchronizes with `stream` (to read the header and the validation result).
 */
awsrc_status awsrc_decode_add(const uint8_t* stream_bytes, uint64_t stream_len, int32_t n_modules,
                              void* const* W0_ptrs, const int64_t* rows, const int64_t* cols,
                              int32_t w0_dtype, void* workspace, size_t* ws_bytes, void* stream);

/* Host-side description of a validated stream, filled by awsrc_decode_prepare. */
typedef struct awsrc_decode_plan {
  int32_t C, P, b, S;
  int32_t idx_bits, seed_bits, L_rec, n_modules;
  int32_t w0_dtype, scale_fmt;
  int64_t K;
  uint64_t T_total;
  uint64_t h;
  const uint8_t* records;   /* device pointer to the first record */
  void* workspace;          /* the workspace the plan's tables live in */
} awsrc_decode_plan;

/*
 * Validation half of awsrc_decode_add: reads and checks the header, checks
 * every record on the device, and builds the basis, module and pointer tables
 * in the workspace (two-phase size query as above; the query itself reads the
 * header and so synchronizes).  Synchronizes with `stream`.  On AWSRC_OK the
 * plan and workspace stay valid for any number of awsrc_decode_apply calls as
 * long as the stream bytes, the workspace and the W0 buffers are unchanged.
 */
awsrc_status awsrc_decode_prepare(const uint8_t* stream_bytes, uint64_t stream_len, int32_t n_modules,
                                  void* const* W0_ptrs, const int64_t* rows, const int64_t* cols,
                                  int32_t w0_dtype, awsrc_decode_plan* plan, void* workspace,
                                  size_t* ws_bytes, void* stream);

/*
 * Apply half of awsrc_decode_add: one asynchronous kernel launch that adds
 * every record of a prepared stream onto W0 (each call adds again).
 */
awsrc_status awsrc_decode_apply(const awsrc_decode_plan* plan, void* stream);

/*
 * Dense bf16 repaired weights, the form the evaluation of Sec. 4 runs on:
 * W_hat = bf16(W0 + R_hat) for every tile, with W0 = f32(q - z) * s
 * recomputed from the stored backbone (the last step of awsrc_backbone_rtn)
 * rather than read from a materialized fp32 W0, and R_hat the stream's
 * corrections (Eq. (1), Sec. 3.2).  Tiles without a record get bf16(W0).
 * The sum is formed in fp32 and rounded once to bf16, nearest even.
 *  plan       prepared by awsrc_decode_prepare with w0_dtype AWSRC_DTYPE_BF16
 *             and W0_ptrs naming the OUTPUT buffers [rows, cols] bf16 of each
 *             module; their contents are never read, every element is written.
 *  group      the backbone group (64, 128 or 256); cols % group == 0.
 *  codes, scale_f16, zero
 *             host arrays [n_modules] of device pointers to each module's
 *             backbone in the layouts awsrc_backbone_rtn writes; codes
 *             8-byte aligned, scale_f16 2-byte aligned.  C >= 16 and at
 *             most 2^36 weights per module.
 * The backbone pointers are staged in the plan's workspace: calls on one plan
 * are ordered by `stream`, and calls on different streams must not share a
 * plan.  Synchronizes with `stream` once (to read the module shapes) before
 * one asynchronous launch.  Errors: AWSRC_EINVAL for a plan that is not
 * prepared or not bf16, a bad group, C < 16, a NULL or misaligned backbone
 * pointer, cols not a multiple of group, or a module over 2^36 weights.
 */
awsrc_status awsrc_reconstruct_bf16(const awsrc_decode_plan* plan, int32_t group,
                                    const uint8_t* const* codes, const uint16_t* const* scale_f16,
                                    const uint8_t* const* zero, void* stream);

/*
 * Dense bf16 repaired weights of several nested prefixes of one stream in one
 * streaming pass (Sec. 3.3: every record-boundary prefix of a ranked stream
 * decodes without refitting; Sec. 4 evaluates each operating point as dense
 * BF16 weights): target o receives W_hat = bf16(W0 + R_hat) with R_hat the
 * correction of the stream's first K_out[o] records only.  The backbone and
 * each record's correction are computed once per pass and written to every
 * target; the result is the same as awsrc_reconstruct_bf16 of each prefix.
 *  plan       prepared by awsrc_decode_prepare on the longest stream (any
 *             w0_dtype: its own W0 buffers are not touched).
 *  n_out      number of targets, 1..8.
 *  K_out      host array [n_out]: records per target, each 0..plan->K (any
 *             order; equal values are allowed).
 *  out_ptrs   host array [n_out * n_modules] of device pointers, target o of
 *             module m at o * n_modules + m: bf16 [rows, cols], 16-byte
 *             aligned, every element written, never read; targets must not
 *             overlap.
 *  group, codes, scale_f16, zero   as for awsrc_reconstruct_bf16.
 * Synchronizes once (module table read-back) before launching; EINVAL on a
 * bad argument (nothing launched).
 */
awsrc_status awsrc_reconstruct_bf16_prefixes(const awsrc_decode_plan* plan, int32_t n_out, const int64_t* K_out,
                                             void* const* out_ptrs, int32_t group, const uint8_t* const* codes,
                                             const uint16_t* const* scale_f16, const uint8_t* const* zero,
                                             void* stream);

/*
 * Dense bf16 repaired weights on the RTN-INT4-SDQ backbone (Sec. 4 evaluates
 * the codecs on RTN-INT4-SDQ as dense BF16 weights): as
 * awsrc_reconstruct_bf16 (n_out == 0) or awsrc_reconstruct_bf16_prefixes
 * (n_out 1..8), with each group's scale the SDQ scale
 * s_hat_g = f32(mu_b + code_g * step_b) of awsrc_backbone_sdq_dequant instead
 * of an fp16 scale, so W0 = f32(q - z) * s_hat exactly as that call writes it.
 *  n_out, K_out, out_ptrs   0 and NULLs: into the plan's own (bf16) W0
 *             buffers with every record; else as for the prefixes call.
 *  sdq_code   host array [n_modules] of device pointers: int8 [rows * cols/group]
 *             (awsrc_sdq_encode's codes of the module's scales, row-major).
 *  sdq_mean, sdq_step   host arrays [n_modules] of device pointers: fp32
 *             [ceil(groups / 256)] each, 4-byte aligned.
 *  group, codes, zero   as for awsrc_reconstruct_bf16.
 * Synchronizes once (module table read-back) before launching; EINVAL on a
 * bad argument (nothing launched).
 */
awsrc_status awsrc_reconstruct_bf16_sdq(const awsrc_decode_plan* plan, int32_t n_out, const int64_t* K_out,
                                        void* const* out_ptrs, int32_t group, const uint8_t* const* codes,
                                        const int8_t* const* sdq_code, const float* const* sdq_mean,
                                        const float* const* sdq_step, const uint8_t* const* zero, void* stream);

/* Host-only helpers (no device needed). */
/* L_rec in bytes for T_total tiles; -1 if p is invalid. */
int64_t awsrc_record_bytes(const awsrc_params* p, int64_t T_total);
/* h = 40 + 8 * n_modules; -1 if n_modules < 1. */
int64_t awsrc_header_bytes(int32_t n_modules);
/* floor(bpw * n_weights / 8) in IEEE double; -1 on invalid input. */
int64_t awsrc_budget_bytes(double bpw, int64_t n_weights);
/* min(n_eligible, (budget_bytes - h) / L_rec); AWSRC_ENOSPC if budget < h, -1 on bad input. */
int64_t awsrc_prefix_K(int64_t budget_bytes, int64_t h, int64_t L_rec, int64_t n_eligible);

#ifdef __cplusplus
}
#endif
#endif /* AWSRC_H */
