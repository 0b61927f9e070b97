/*
 * pot_attn.h -- C ABI of libpotattn: single-token decode attention over a key
 * cache stored as signed power-of-two (PoT) fixed-point codes, for AMD MI355X
 * (gfx950).
 *
 * Method: "Shift-Accumulate Attention: Multiplier-Free Query-Key Products for
 * Transformer Decoding" (arXiv 2609.09208).
 *   - key code and query quantiser ............ Sec. II-A, eq. (pot)
 *   - shift-accumulate (SAC) score ............. Sec. II-B, eq. (sac)
 *   - exactness by head-room F >= E ............ Sec. II-C, eq. (exact)
 *   - mantissa family PoT-Mk ................... Sec. II-D, eq. (mant)
 *   - integer-log2 online softmax max .......... Sec. II-E, eq. (logsm)
 *   - fused split decode kernel, code-only cache Sec. II-F
 *   - Hadamard (score-preserving) rotation ..... Sec. I-A and Sec. V-A
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All tensor pointers are DEVICE pointers (hipMalloc'd or torch-owned
 *    device memory) unless the argument says "host". The caller owns every
 *    buffer; the library never allocates or frees device memory.
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t passed as
 *    void*, NULL = the legacy default stream). No entry point synchronises
 *    the host.
 *  - Every argument check runs on the host before any HIP call, so invalid
 *    arguments return an error without touching the GPU. Errors are returned,
 *    never thrown; pot_last_error() gives a human-readable detail for the
 *    calling thread.
 *  - Inputs are read-only; outputs must not alias inputs. Codes, V, K and q
 *    pointers must be 16-byte aligned.
 *  - Head dimension d is 64.
 *
 * Key cache layout ("row" = one (batch b, kv-head h, position t)):
 *    row(b, h, t) = (b * Hkv + h) * t_cap + t,   0 <= t < t_cap
 *  codes_se  uint8 [rows][d/2]   sign/exponent nibbles. Byte i holds element
 *                                2i in its low nibble and 2i+1 in its high
 *                                nibble. nibble = (neg << 3) | e with
 *                                e in 0..E a magnitude 2^-e and e = E+1 = 7
 *                                the exact zero (stored with neg = 0, j = 0).
 *  codes_m   uint8 [rows][8*k]   k mantissa bit-planes of 64 bits each
 *                                (little-endian). Bit m of plane b is bit b of
 *                                the mantissa j_m of element m. NULL if k = 0.
 *  key_scale float [rows]        per-key-vector scale s_j (Sec. II-A).
 *  v_cache   fp16                value cache, token-interleaved in groups of
 *                                8: token t, dim m of sequence q = b*Hkv + h
 *                                is the half at
 *                                  (q*t_cap + (t/8)*8) * d + m*8 + t%8,
 *                                so 8 consecutive tokens of one dim are one
 *                                16-byte word (the matrix-core operand of the
 *                                A.V product). Written by pot_store_values.
 *                                t_cap must be a multiple of 8.
 *
 * Decoded key element (eq. pot and eq. mant):
 *    K^_m = s * sigma_m * (1 + j_m / 2^k) * 2^-e_m,   or 0 for the zero code.
 */
#ifndef POT_ATTN_H
#define POT_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define POT_HEAD_DIM 64
#define POT_ABI_VERSION 1

typedef enum pot_status {
  POT_OK = 0,
  POT_ERR_INVALID_ARG = 1, /* null pointer, bad size, F < E, T out of range  */
  POT_ERR_UNSUPPORTED = 2, /* d != 64, unsupported field widths, head map     */
  POT_ERR_WORKSPACE = 3,   /* workspace too small                             */
  POT_ERR_HIP = 4          /* a HIP runtime or launch error (see last_error)  */
} pot_status;

/* Key-code format (Sec. II-A, II-D).
 *  head_dim  : d, must be 64.
 *  exp_bits  : exponent field width; only 3 is supported, giving E = 6 and the
 *              field value 7 as exact zero (b = 4 bits with the sign).
 *  mant_bits : k in 0..4. 0 is PoT-4, k > 0 is PoT-Mk (4 + k stored bits).
 *  frac_bits : fixed-point head-room F of eq. (sac). Must satisfy F >= E
 *              (eq. exact: every shift F - e is then a non-negative left shift)
 *              and F <= 12 (keeps the int32 accumulator exact for k <= 4).
 *              The paper's example is F = 7.
 *  hadamard  : 1 to rotate keys and queries by the orthonormal 64x64
 *              Sylvester-Hadamard matrix H/8 before quantisation; 0 otherwise.
 */
typedef struct pot_format {
  int32_t head_dim;
  int32_t exp_bits;
  int32_t mant_bits;
  int32_t frac_bits;
  int32_t hadamard;
} pot_format;

/* Optional debug taps of pot_decode_attention, pot_ds4a_decode_attention and
 * pot_int8_decode_attention.
 * Every pointer may be NULL (tap off). When any tap is non-NULL the call runs
 * an instrumented build of the same kernel source.
 *  qhat     int8  [B][Hq][d]  quantised (rotated) query q^ (eq. pot)
 *  delta    float [B][Hq]     query step Delta_i
 *  scores   int32 [B][Hq][T]  exact integer accumulator of eq. (sac) at
 *                             head-room F (for k > 0 at scale 2^-(F+k))
 *  m_final  int32 [B][Hq]     integer log2-domain maximum M of eq. (logsm)
 *  m_split  int32 [B][Hq][n_splits] per-split maxima
 *  force_splits (in)  if > 0, use this many key splits instead of the planner
 *  n_splits     (out) the number of key splits used (written on the host)
 *  split_len    (out) keys per split (the last split may be shorter)
 *  decode_begin, decode_end (in) NULL, or hipEvent_t handles the caller
 *               created: the call records decode_begin on its stream right
 *               before the decode kernel and decode_end right after it (before
 *               the split combine), so that kernel can be timed alone. They
 *               do not select the instrumented build. A failed record returns
 *               POT_ERR_HIP.
 *  force_wg_waves (in) 0: the planner picks the decode workgroup size; 4:
 *               four-wave workgroups, each wave taking every fourth 64-key
 *               tile of its split; or the wave count of the engine's
 *               CU-wide variant: one workgroup per CU whose waves claim the
 *               split's tiles from a counter in LDS (shift-accumulate
 *               kernels, fp16 or INT8 values: 16 at k <= 2, 12 at k = 3
 *               and 4; decoded-code engines: 16, or 12 for PoT-4 bytes over
 *               fp16 values or with power-of-two weights; INT8 comparator:
 *               12; the fp16 comparator has none). Other values return
 *               POT_ERR_INVALID_ARG. Scores and maxima do not
 *               depend on it; O does to fp32 rounding (with claimed tiles the
 *               order of the sums varies from call to call).
 *  wg_waves     (out) the waves per workgroup used (written on the host)
 */
typedef struct pot_debug {
  int8_t* qhat;
  float* delta;
  int32_t* scores;
  int32_t* m_final;
  int32_t* m_split;
  int32_t force_splits;
  int32_t n_splits;
  int32_t split_len;
  void* decode_begin;
  void* decode_end;
  int32_t force_wg_waves;
  int32_t wg_waves;
} pot_debug;

/* Static string for a status code. Never NULL. */
const char* pot_status_string(pot_status status);

/* Detail of the last error raised on the calling thread ("" if none). */
const char* pot_last_error(void);

/* Bytes of codes_se + codes_m per cache row for `fmt` (32 + 8k for d = 64),
 * or 0 if the format is invalid. Host-only, no HIP call. */
size_t pot_code_bytes_per_row(const pot_format* fmt);

/* Encode fp16 keys to PoT / PoT-Mk codes (Sec. II-A, II-D).
 *  k_fp16         [n_rows][d] fp16, dense, device.
 *  n_rows         number of key vectors (>= 0; 0 is a no-op).
 *  out_row_stride output row r is written at cache row r * out_row_stride
 *                 (1 for a dense block; t_cap to append one token to each of
 *                 n_rows sequences, with the output pointers offset by t rows).
 *  scale_mode     0: s = max_m |K'_m| (per key vector, written to key_scale);
 *                 1: s is read from key_scale (caller-given, e.g. one value
 *                    per head); ratios above the top code saturate.
 *  Per element: u = fl32(|K'_m| / s), rounded to the grid value
 *  (1 + j/2^k) 2^-e nearest in log2 distance; u below 2^-(E+1/2) becomes the
 *  exact zero code. K' = K, or fl32(H K / 8) when fmt->hadamard.
 *  codes_se [rows][32], codes_m [rows][8k] (NULL iff k = 0), key_scale [rows].
 */
pot_status pot_encode_keys(const pot_format* fmt, const uint16_t* k_fp16,
                           int64_t n_rows, int64_t out_row_stride,
                           int32_t scale_mode, float* key_scale,
                           uint8_t* codes_se, uint8_t* codes_m, void* stream);

/* Store fp16 values into the token-interleaved value cache.
 *  v_fp16   [n_seq][n_tok][d] fp16, dense, device (token-major rows).
 *  n_seq    sequences (b*Hkv + h order, consecutive from v_cache).
 *  n_tok    tokens per sequence to write, at positions t0 .. t0+n_tok-1
 *           (n_tok = 1 appends one decoded token).
 *  t_cap    cache capacity per sequence, a positive multiple of 8.
 *  Tokens outside [t0, t0+n_tok) are left untouched. Errors: negative sizes,
 *  t_cap not a multiple of 8, the range outside [0, t_cap), NULL or
 *  misaligned pointers (INVALID_ARG). */
pot_status pot_store_values(const uint16_t* v_fp16, int64_t n_seq, int64_t n_tok,
                            int64_t t_cap, int64_t t0, uint16_t* v_cache,
                            void* stream);

/* Store fp16 values as INT8 codes with a power-of-two per-token scale
 * (Sec. II-E, the value cache the paper pairs with PoT keys: 64 + 1 bytes per
 * token instead of 128). The paper leaves the rounding open; here, per token
 * row v (d values): g = the largest integer with max|v| 2^g <= 127 (g = 0 for
 * an all-zero row) and v^ = round-half-even(v 2^g), so |v^| <= 127 and the
 * value is v^ 2^-g (exact for every fp16 input range: g lies in [-10, 30]).
 *  v_fp16   [n_seq][n_tok][d] fp16, dense, device (token-major rows).
 *  v_u8     value bytes v^ + 128 (offset binary), token-interleaved like the
 *           fp16 cache: byte ((t/8)*8)*d + dim*8 + t%8 of each sequence's
 *           t_cap*d bytes; [B*Hkv][t_cap][d] bytes in all.
 *  v_exp    int8 [B*Hkv][t_cap]: g of each token.
 * n_seq, n_tok, t_cap, t0 and the errors as pot_store_values (all three
 * pointers 16-byte aligned). */
pot_status pot_store_values_int8(const uint16_t* v_fp16, int64_t n_seq, int64_t n_tok,
                                 int64_t t_cap, int64_t t0, uint8_t* v_u8,
                                 int8_t* v_exp, void* stream);

/* Workspace bytes pot_decode_attention needs for this problem shape: the
 * prepared query operands of each (batch, kv head) and the key-split partials
 * (M_s, l_s, o_s) for the largest split count the planner can choose.
 * Host-only. Returns 0 for invalid shapes. The same figure serves
 * pot_int8_decode_attention and pot_fp16_decode_attention. */
size_t pot_decode_workspace_bytes(int32_t B, int32_t Hq, int32_t Hkv,
                                  int32_t T);

/* Workspace bytes for a given split count (as forced through
 * pot_debug.force_splits; the count is clamped as the decode call clamps it).
 * Host-only. Returns 0 for invalid shapes. */
size_t pot_decode_workspace_bytes_for_splits(int32_t B, int32_t Hq, int32_t Hkv,
                                             int32_t T, int32_t n_splits);

/* Zero a workspace (a fill kernel on `stream`). Optional: the decode calls
 * need no particular initial workspace contents. */
pot_status pot_workspace_init(void* workspace, size_t ws_bytes, void* stream);

/* Single-token decode attention with PoT keys (Sec. II-B, II-E, II-F).
 *  q            [B][Hq][d] fp32 query (post-RoPE).
 *  codes_se, codes_m, key_scale, v_cache: cache as laid out above, t_cap
 *               rows per (b, kv-head) sequence (t_cap a multiple of 8).
 *  kv_head_of_q HOST int32 [Hq]: kv head serving each query head (GQA). Every
 *               kv head must serve the same number G = Hq/Hkv of query heads,
 *               G in {1, 2, 4, 8}.
 *  T            keys attended, 1 <= T <= t_cap and T <= 2^24 - 8
 *               (POT_ERR_UNSUPPORTED above: the kernel addresses a
 *               sequence's rows with 32-bit byte offsets).
 *  out          [B][Hq][d] fp32: O = softmax(S^ / sqrt(d)) V.
 *  workspace    >= pot_decode_workspace_bytes(B, Hq, Hkv, T) bytes, 256-byte
 *               aligned. Calls that share a workspace must not overlap in
 *               time.
 * Steps: q is rotated (if hadamard) and quantised to int8 with step
 * Delta = amax/127; each score is the exact int32 sum of sign-flipped
 * shifts of q^ (eq. sac: the products q^ 2^(F-e) are formed by packed 16-bit
 * arithmetic shifts of q^ 2^7; the signs and the sum are applied by
 * v_dot2_i32_i16, the dot unit's multiply-add, with weights +-1, 0 for the
 * zero code; PoT-Mk adds one such sum per mantissa bit plane, combined
 * by shifts); x = acc * s * Delta * log2(e) * 2^-(F+k) / 8 in a fixed fp32
 * order; the running maximum is the integer M = ceil(max x)
 * (eq. logsm) so rescales are exact powers of two; weights 2^(x-M) multiply
 * the fp16 values with fp32 accumulation (matrix cores, weights split into
 * fp16 high and low parts); key splits (chosen to fill the GPU's resident
 * workgroup slots in one round) are merged with exact 2^(M_s - M) factors.
 * Launches: a query-preparation kernel, the split decode kernel and, with
 * more than one split, a combine kernel, all on `stream`.
 */
pot_status pot_decode_attention(const pot_format* fmt, const float* q,
                                const uint8_t* codes_se,
                                const uint8_t* codes_m, const float* key_scale,
                                const uint16_t* v_cache, int64_t t_cap,
                                const int32_t* kv_head_of_q, int32_t B,
                                int32_t Hq, int32_t Hkv, int32_t T, float* out,
                                void* workspace, size_t ws_bytes,
                                pot_debug* dbg, void* stream);

/* One decode step on a cache that holds only codes (Sec. II-F, Sec. V-F): the
 * new token of every (b, kv-head) sequence is appended at position T - 1 and
 * attention then runs over positions 0 .. T-1, in one call. Equivalent to
 * pot_encode_keys(fmt, k_new, B*Hkv, t_cap, 0, ...) on the rows at T - 1,
 * pot_store_values(v_new, B*Hkv, 1, t_cap, T - 1, v_cache) and
 * pot_decode_attention(...) over T keys, with bit-identical cache contents and
 * output, but without the two extra launches: the query-preparation kernel
 * writes the new rows before the decode kernel starts.
 *  k_new, v_new [B][Hkv][d] fp16, dense, device, 16-byte aligned: the new
 *               token's key (encoded with the row absmax scale, rotated first
 *               when fmt->hadamard) and values.
 *  codes_se, codes_m, key_scale, v_cache: the cache as for
 *               pot_decode_attention, written at row T - 1 of each sequence
 *               (nothing else is written).
 *  Other arguments, the workspace, debug taps (the scores include the new
 *  key) and errors as pot_decode_attention; NULL or misaligned k_new / v_new
 *  -> INVALID_ARG. Inputs q, k_new and v_new may not alias the cache. */
pot_status pot_append_decode_attention(const pot_format* fmt, const float* q,
                                       const uint16_t* k_new, const uint16_t* v_new,
                                       uint8_t* codes_se, uint8_t* codes_m,
                                       float* key_scale, uint16_t* v_cache,
                                       int64_t t_cap, const int32_t* kv_head_of_q,
                                       int32_t B, int32_t Hq, int32_t Hkv, int32_t T,
                                       float* out, void* workspace, size_t ws_bytes,
                                       pot_debug* dbg, void* stream);

/* Decode attention with PoT keys and INT8 values (pot_store_values_int8):
 * O = sum_t p_t v^_t 2^-g_t / sum_t p_t with the weights p of
 * pot_decode_attention (Sec. II-E). engine 0 scores by shift-accumulate as
 * pot_decode_attention, engine 1 by the byte-decode path of
 * pot_ds4a_decode_attention (PoT-4 only, else POT_ERR_UNSUPPORTED); the
 * int32 scores and integer maxima are the same as with fp16 values. In the
 * kernel each workgroup takes g_ref = min g over its keys and forms the
 * weights p 2^(g_ref - g_t) (exact, never above p) for the matrix cores,
 * with the value bytes read as the fp16 numbers 1152 + v^; the 1152 offset
 * and 2^-g_ref are applied to the fp32 sums. Arguments, workspace, taps and
 * errors as pot_decode_attention, with (v_u8, v_exp) in place of v_cache
 * (NULL or not 16-byte aligned -> INVALID_ARG); engine outside {0, 1} ->
 * INVALID_ARG. */
pot_status pot_decode_attention_v8(const pot_format* fmt, int32_t engine, const float* q,
                                   const uint8_t* codes_se, const uint8_t* codes_m,
                                   const float* key_scale, const uint8_t* v_u8,
                                   const int8_t* v_exp, int64_t t_cap,
                                   const int32_t* kv_head_of_q, int32_t B, int32_t Hq,
                                   int32_t Hkv, int32_t T, float* out, void* workspace,
                                   size_t ws_bytes, pot_debug* dbg, void* stream);

/* Both products by powers of two (Sec. II-E, the option eq. logsm and eq. av
 * describe): the scores as pot_decode_attention_v8 (engine 0 or 1), INT8
 * values, and the power-of-two weights A~_t = 2^-k_t of eq. logsm in place
 * of the softmax weights: k_t = M - ceil(x_t - 1/2) (M - x_t rounded half up,
 * so a rising running maximum rescales every earlier weight exactly), and
 * O = sum_t A~_t v^_t 2^-g_t / sum_t A~_t (eq. av leaves the normalisation
 * out; no k_max cut: weights below 2^-36 of the largest vanish in the fp16
 * weight operand). Every product A~_t v^_t 2^-g_t is exact; the sums are fp32
 * on the matrix cores. Arguments, layout, workspace, taps and errors as
 * pot_decode_attention_v8. */
pot_status pot_decode_attention_v8_pow2(const pot_format* fmt, int32_t engine,
                                        const float* q, const uint8_t* codes_se,
                                        const uint8_t* codes_m, const float* key_scale,
                                        const uint8_t* v_u8, const int8_t* v_exp,
                                        int64_t t_cap, const int32_t* kv_head_of_q,
                                        int32_t B, int32_t Hq, int32_t Hkv, int32_t T,
                                        float* out, void* workspace, size_t ws_bytes,
                                        pot_debug* dbg, void* stream);

/* pot_append_decode_attention on a cache with INT8 values: the new token's
 * values are quantised as by pot_store_values_int8 and stored with their
 * exponent at position T - 1, then pot_decode_attention_v8 runs with the
 * given engine over T keys, in one call (the cache holds only codes: 32 + 4 +
 * 65 bytes per PoT-4 key). Arguments and errors as the two calls it
 * combines. */
pot_status pot_append_decode_attention_v8(const pot_format* fmt, int32_t engine,
                                          const float* q, const uint16_t* k_new,
                                          const uint16_t* v_new, uint8_t* codes_se,
                                          uint8_t* codes_m, float* key_scale,
                                          uint8_t* v_u8, int8_t* v_exp, int64_t t_cap,
                                          const int32_t* kv_head_of_q, int32_t B,
                                          int32_t Hq, int32_t Hkv, int32_t T, float* out,
                                          void* workspace, size_t ws_bytes,
                                          pot_debug* dbg, void* stream);

/* Bytes of the static device scratch behind pot_decode_attention_noalloc
 * (one copy per GPU, held until the process ends). */
#define POT_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)

/* pot_decode_attention for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same computation, kernels and arguments, without the
 * workspace arguments. The workspace is a static device array of
 * POT_NOALLOC_SCRATCH_BYTES per GPU that the library owns; the call allocates
 * nothing (no hipMalloc, no hipFree). Its device address is looked up once
 * per GPU, on the first call with that GPU current; `stream` must belong to
 * the current GPU.
 * Errors: as pot_decode_attention; a shape whose workspace bound
 * (pot_decode_workspace_bytes, or pot_decode_workspace_bytes_for_splits with
 * dbg->force_splits) exceeds POT_NOALLOC_SCRATCH_BYTES -> POT_ERR_WORKSPACE,
 * checked on the host before any HIP call. The bound covers the largest split
 * count the planner may choose: 264 bytes per query head and key split (the
 * split partials) plus one prepared-query slot per kv head and key split
 * (1280 bytes at G = 8). At the TinyLlama shape (Hq = 32, Hkv = 4) it is
 * about 7 MB for B >= 8 and 1.7 MB at B = 1.
 * Every call on one GPU shares that GPU's scratch, which keeps the previous
 * call's contents (the kernels write every word they read, so nothing needs
 * clearing): calls that overlap in time on one GPU race and must not be made. */
pot_status pot_decode_attention_noalloc(const pot_format* fmt, const float* q,
                                        const uint8_t* codes_se, const uint8_t* codes_m,
                                        const float* key_scale, const uint16_t* v_cache,
                                        int64_t t_cap, const int32_t* kv_head_of_q, int32_t B,
                                        int32_t Hq, int32_t Hkv, int32_t T, float* out,
                                        pot_debug* dbg, void* stream);

/* ---- comparison paths on the same cache skeleton --------------------- */

/* INT8 uniform key codes (the multiply-accumulate comparator of Sec. III and
 * Sec. VI): per key vector s = amax/127, k^ = clamp(rne(K' * (127/amax))).
 *  codes int8 [rows][d], key_scale float [rows]. hadamard as in pot_format. */
pot_status pot_int8_encode_keys(const uint16_t* k_fp16, int64_t n_rows,
                                int64_t out_row_stride, int32_t hadamard,
                                float* key_scale, int8_t* codes, void* stream);

/* Decode attention with INT8 keys: scores by 4-way int8 dot products
 * (v_dot4), the same query quantiser, integer-M softmax and fp16 A.V. */
pot_status pot_int8_decode_attention(
    const float* q, const int8_t* codes, const float* key_scale,
    const uint16_t* v_cache, int64_t t_cap, const int32_t* kv_head_of_q,
    int32_t B, int32_t Hq, int32_t Hkv, int32_t T, int32_t hadamard,
    float* out, void* workspace, size_t ws_bytes, pot_debug* dbg,
    void* stream);

/* Decode attention over a PoT-4 cache (mant_bits = 0) with the score computed
 * by a software form of the packed shift-dot operation DS4A (Sec. III,
 * eq. ds4a): each code nibble is decoded by a byte table (v_perm_b32) to the
 * int8 value sigma 2^(6-e) (0 for the zero code, which must be stored with
 * neg = 0 as pot_encode_keys writes it), and v_dot4_i32_i8 accumulates
 * q^ * sigma 2^(6-e); one left shift by F - 6 gives exactly the int32 score
 * of pot_decode_attention. This is a multiply path, provided to measure what
 * a packed shift-dot would buy (eq. proj); pot_decode_attention is the
 * shift-accumulate path. Arguments, layout, workspace, taps and errors as
 * pot_decode_attention; fmt->mant_bits other than 0 -> POT_ERR_UNSUPPORTED. */
pot_status pot_ds4a_decode_attention(const pot_format* fmt, const float* q,
                                     const uint8_t* codes_se, const float* key_scale,
                                     const uint16_t* v_cache, int64_t t_cap,
                                     const int32_t* kv_head_of_q, int32_t B,
                                     int32_t Hq, int32_t Hkv, int32_t T, float* out,
                                     void* workspace, size_t ws_bytes,
                                     pot_debug* dbg, void* stream);

/* Decode attention over a PoT or PoT-Mk cache with the codes decoded to
 * integer weights and scored on the dot unit (a multiply path beside the
 * shift-accumulate one, Sec. III, eq. ds4a and eq. mant): PoT-4 as
 * pot_ds4a_decode_attention (bytes sigma 2^(6-e), v_dot4_i32_i8); PoT-Mk as
 * 16-bit weights sigma (2^k + j) 2^(7-e) (0 for the zero code), at most
 * 31 * 128, with v_dot2_i32_i16 over q^ for two elements per head, one dot
 * per head and element pair whatever k. The int32 scores, integer maxima and
 * outputs equal pot_decode_attention's (same scores tap convention, 2^-(F+k)
 * for k > 0). Arguments, layout, workspace, taps and errors as
 * pot_decode_attention. */
pot_status pot_dot_decode_attention(const pot_format* fmt, const float* q,
                                    const uint8_t* codes_se, const uint8_t* codes_m,
                                    const float* key_scale, const uint16_t* v_cache,
                                    int64_t t_cap, const int32_t* kv_head_of_q, int32_t B,
                                    int32_t Hq, int32_t Hkv, int32_t T, float* out,
                                    void* workspace, size_t ws_bytes, pot_debug* dbg,
                                    void* stream);

/* Decode attention on an unquantised fp16 cache (the FP16 baseline of
 * Sec. IV): q is rounded to fp16, scores accumulate in fp32.
 *  k_fp16 [rows][d] fp16 row-major keys; v_cache as above. */
pot_status pot_fp16_decode_attention(const float* q, const uint16_t* k_fp16,
                                     const uint16_t* v_cache, int64_t t_cap,
                                     const int32_t* kv_head_of_q, int32_t B,
                                     int32_t Hq, int32_t Hkv, int32_t T,
                                     float* out, void* workspace,
                                     size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* POT_ATTN_H */
