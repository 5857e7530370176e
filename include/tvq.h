/*
 * tvq.h -- C ABI of the TurboAngle KV-cache codec for AMD Instinct MI355X (gfx950).
 *
 * Method: TurboAngle (arXiv 2603.27467).  Each (token, head) K or V vector x of length d is
 *   1. sign-flipped by a random +-1 diagonal D and transformed by the normalized fast
 *      Walsh-Hadamard transform H (section 2; Algorithm 1, first step);
 *   2. split into d/2 consecutive pairs, each written in polar form (r_i, theta_i) with
 *      theta_i quantized to one of n uniform bins (Algorithm 1), n chosen per layer and
 *      separately for K and V (section 3.2, per-layer MixedKV / early-boost);
 *   3. its pair norms kept in fp32 or quantized per vector by min-max scalar quantization,
 *      linear (eq. (2)) or in log space (section 3.3), with the vector's min and max stored
 *      as two fp32 values;
 *   4. bit-packed into the compressed cache.
 * Decoding rebuilds y^ = r^ (cos 2 pi k/n, sin 2 pi k/n) and x^ = D H y^ (section 3.1,
 * reconstruction), using H^-1 = H and D^-1 = D.
 *
 * Conventions for every entry point:
 *   - Plain C types only.  Device pointers are HIP device memory owned by the caller.
 *     `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *   - Nothing here allocates device memory except tvq_create; tvq_encode / tvq_decode only
 *     validate on the host and enqueue kernels on `stream`, then return without waiting.
 *   - Argument errors are reported synchronously by the return value and nothing is
 *     launched.  A launch failure returns TVQ_ERR_HIP.  Faults inside a kernel surface at the
 *     caller's next synchronization, as for any HIP work.
 *   - A codec handle is immutable after tvq_create; concurrent calls on different streams are
 *     safe.  Ordering an encode and a decode that touch the same cache tokens is the caller's
 *     job (stream order or events).
 */
#ifndef TVQ_H
#define TVQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TVQ_ABI_VERSION 3
#define TVQ_MAX_LAYERS 256

typedef enum {
  TVQ_OK = 0,
  TVQ_ERR_INVALID_ARG = -1,  /* a pointer, size, stride, alignment or config value is bad */
  TVQ_ERR_UNSUPPORTED = -2,  /* valid for the method but not built for the GPU (e.g. d=32) */
  TVQ_ERR_HIP = -3,          /* a HIP runtime call or kernel launch failed */
  TVQ_ERR_ALLOC = -4,        /* tvq_create could not allocate its device tables */
  TVQ_ERR_SCRATCH = -5       /* the call needs more scratch than the library's static buffer
                                holds (tvq_attention_decode_noalloc) */
} tvq_status;

typedef enum { TVQ_BF16 = 0, TVQ_F32 = 1 } tvq_dtype;

/* Norm storage (section 3.3): fp32 norms (16 bits per element, section 3.1 "Rate
 * accounting"), per-vector min-max linear (eq. (2)), or min-max on log r (log-space variant). */
typedef enum { TVQ_NORM_F32 = 0, TVQ_NORM_LINEAR = 1, TVQ_NORM_LOG = 2 } tvq_norm_mode;

/* One layer of the per-layer codebook table (section 3.2: an independent (n_K, n_V) per
 * layer; section 3.3: K and V norm bits, e.g. K 8-bit linear / V 4-bit log).
 *   n_k, n_v           angle bins, 2..4096 (stored in ceil(log2 n) bits per pair)
 *   norm_bits_k/_v     1..16 for LINEAR/LOG; ignored (32) for F32
 *   norm_mode_k/_v     tvq_norm_mode                                                  */
typedef struct {
  uint16_t n_k, n_v;
  uint8_t norm_bits_k, norm_bits_v;
  uint8_t norm_mode_k, norm_mode_v;
} tvq_layer_cfg;

/* Codec configuration.
 *   num_layers  L, 1..TVQ_MAX_LAYERS;  num_heads  H (KV heads) >= 1;
 *   head_dim    d; the GPU kernels are built for d = 64 and d = 128
 *   layers      [L] table, copied by tvq_create
 *   signs       optional host array of +-1 (int8): [L][d], or [d] when shared_signs != 0.
 *               NULL: drawn from `seed` with SplitMix64 (Steele, Lea and Flood 2014) as
 *               tvq_make_signs describes.  The paper samples D once from a seeded PRNG and
 *               shares it across layers (section 3.1 "Implementation"); shared_signs = 1 gives
 *               that, shared_signs = 0 draws an independent D per layer.
 *   angle_packing  0: every angle code in ceil(log2 n) bits; 1: group packing for a
 *               non-power-of-two n (the paper counts log2(n)/2 bits per element, section 3.1
 *               "Rate accounting"): groups of g = 8 codes (g = 4 for n > 255) stored as the
 *               base-n number sum_i c_(g*j+i) n^i in W = ceil(log2(n^g)) bits, group j at bits
 *               [j*W, (j+1)*W) of the record.  n = 48 takes 45 bytes per d = 128 vector
 *               instead of 48.  Powers of two are stored the same way under both settings. */
typedef struct {
  int32_t num_layers, num_heads, head_dim;
  int32_t shared_signs;
  uint64_t seed;
  const tvq_layer_cfg* layers;
  const int8_t* signs;
  int32_t angle_packing;
} tvq_config;

/* A strided [L][B][H][T][d] view of K and V (the same strides for both), in elements, with
 * d contiguous.  `batch` = B, `tokens` = T of this call.  Every vector must start on a 16-byte
 * boundary (base pointers and strides x element size multiples of 16).  Strides are
 * non-negative; stride_b, stride_h and stride_t are below 2^32, and B*H*T below 2^31.     */
typedef struct {
  int64_t batch, tokens;
  int64_t stride_l, stride_b, stride_h, stride_t;
} tvq_tensor_desc;

/* Compressed cache layout (this project's; the paper only counts bits, section 3.1 "Rate
 * accounting" and eq. (3)).  For each layer l and kind (0 = K, 1 = V) there are three planes:
 *   plane 0  angle codes   P*ceil(log2 n)/8 bytes per vector (P = d/2 pairs), or with group
 *                          packing (P/g)*W/8, rounded up to whole bytes
 *   plane 1  norm data     P*b/8 bytes (LINEAR/LOG codes) or 4P bytes (fp32 norms)
 *   plane 2  header        8 bytes (fp32 r_min, r_max), absent (0 bytes) for fp32 norms
 * Each plane holds B*H*capacity records indexed ((b*H + h)*capacity + t).  Planes follow each
 * other in (layer, kind, plane) order with no padding.  Inside a record, code i occupies bits
 * [i*w, (i+1)*w) of an LSB-first bitstream (bit j is bit j%8 of byte j/8).                */
typedef struct {
  int64_t total_bytes;
  int64_t batch, capacity_tokens;
  int64_t off[TVQ_MAX_LAYERS][2][3];        /* byte offset of each plane */
  int32_t rec_bytes[TVQ_MAX_LAYERS][2][3];  /* bytes per vector in each plane */
} tvq_layout;

typedef struct tvq_codec tvq_codec;

/* Create a codec: validates `cfg`, builds the sign table, the per-(layer, kind) parameters
 * and the reconstruction cos/sin tables (section 3.1, "trigonometric lookup") and uploads
 * them to the current HIP device, whose compute-unit count and attention-kernel occupancy it
 * records for the attention chunk plan.  *out receives the handle (NULL on error).
 * Returns TVQ_ERR_INVALID_ARG (bad config), TVQ_ERR_UNSUPPORTED (d not 64/128),
 * TVQ_ERR_ALLOC or TVQ_ERR_HIP. */
tvq_status tvq_create(const tvq_config* cfg, tvq_codec** out);

/* Free a codec and its device tables (NULL is ignored).  Waits for nothing: the caller must
 * not destroy a codec while its kernels may still run. */
void tvq_destroy(tvq_codec* c);

/* Fill *out with the layout of a cache for `batch` sequences of `capacity_tokens` slots.
 * Host-only; the caller allocates out->total_bytes of device memory (any 16-byte aligned
 * buffer) and passes the same layout to tvq_encode / tvq_decode. */
tvq_status tvq_cache_layout(const tvq_codec* c, int64_t batch, int64_t capacity_tokens,
                            tvq_layout* out);

/* Encode (Algorithm 1 + section 3.3) K and V, each described by `in` with `in_dtype`
 * elements, into cache slots [t_begin, t_begin + in->tokens) of every (layer, batch, head).
 * Requires in->batch == lay->batch and t_begin + in->tokens <= lay->capacity_tokens.
 * k, v: device pointers; cache: device pointer to lay->total_bytes bytes.
 * Launches up to two kernels on `stream` (one for bf16 input of the layers whose formats have a
 * dedicated kernel, one for the rest), twice over for bf16 input of at least 2^19 vectors per
 * kind whose token count is not a multiple of the tile's (16 tokens at d = 128, 32 at d = 64):
 * its whole tiles first, then the remaining tokens; in->tokens == 0 launches nothing. */
tvq_status tvq_encode(const tvq_codec* c, tvq_dtype in_dtype, const void* k, const void* v,
                      const tvq_tensor_desc* in, int64_t t_begin, void* cache,
                      const tvq_layout* lay, void* stream);

/* tvq_encode for bf16 input at d = 128 with a different transform schedule, for comparison:
 * in the layers whose formats have the dedicated kernel (n = 64/256, 8-bit linear or 4-bit
 * log norms), the butterfly stages over element bits 0, 1, 5 and 6 run as one 16-point
 * Hadamard product per 16 vectors on the matrix cores (bf16 operands, fp32 accumulation) and
 * the other three stages follow in registers.  Every stage of W is applied, but not in the
 * canonical ascending order, so a code can differ from tvq_encode's where rounding moves the
 * angle or norm coordinate across a bin boundary (inside the 1e-6-of-range flag zone of the
 * parity rule); other layers are encoded as by tvq_encode.  TVQ_ERR_UNSUPPORTED for d != 128. */
tvq_status tvq_encode_mfma(const tvq_codec* c, const void* k, const void* v,
                           const tvq_tensor_desc* in, int64_t t_begin, void* cache,
                           const tvq_layout* lay, void* stream);

/* Decode (section 3.1, reconstruction) cache slots [t_begin, t_end) of every (layer, batch,
 * head) into k_out / v_out, described by `out` (out->tokens == t_end - t_begin,
 * out->batch == lay->batch), as `out_dtype` (bf16 rounded to nearest even, or fp32).
 * Launches up to two kernels on `stream` (one for the layers whose formats have a dedicated
 * kernel, one for the rest), twice over when a range of at least 2^19 vectors per kind has a
 * token count that is not a multiple of the tile's (16 tokens at d = 128, 32 at d = 64): its
 * whole tiles first, then the remaining tokens; an empty range launches nothing. */
tvq_status tvq_decode(const tvq_codec* c, const void* cache, const tvq_layout* lay,
                      int64_t t_begin, int64_t t_end, tvq_dtype out_dtype, void* k_out,
                      void* v_out, const tvq_tensor_desc* out, void* stream);

/* Attention of one query token per sequence over one layer of the cache -- the consumer of
 * the decoded keys and values, computed from the codes without writing them (standard
 * attention, not part of the paper):
 *   o[b][h*G + g] = sum_{t < t_end} p_t v^_t / sum_t p_t,   p_t = exp(s_t - max_t s_t),
 *   s_t = scale * (q[b][h*G + g] . k^_t),
 * where k^_t, v^_t are the vectors tvq_decode would return for (layer, b, KV head h, t) and
 * G = num_q_heads / H query heads share each KV head.  Because H D is orthogonal (section 2),
 * s_t = scale * (W D q) . y'_t and o = D W (sum_t p_t y'_t) / sum_t p_t with y' the
 * reconstructed pair coordinates (section 3.1): one transform per query and per output.
 *   q, o       device [B][num_q_heads][d], contiguous, bf16 or fp32, 16-byte aligned;
 *              B = lay->batch
 *   t_end      1 .. lay->capacity_tokens tokens attended (slots [0, t_end))
 *   workspace  device scratch of at least tvq_attention_workspace(...) bytes, 16-byte
 *              aligned, owned by the caller; its contents are overwritten
 * The token range is split into equal chunks (whole tile pairs, at least 4 tiles) so that a
 * launch has about one chunk wave per wave slot of the codec's device (its compute units
 * times the resident waves per compute unit of the chunk kernel of the layer's formats, taken
 * at tvq_create); the workspace holds one partial (max, sum, d accumulators) per query head
 * and chunk, so its size depends on the device the codec was created on.
 * tvq_attention_workspace names no layer and gives the size for the formats with the most
 * chunks, which covers every layer.  Query heads are processed up to 4 per pass over the
 * codes (G > 4 reads them ceil(G/4) times).  Arithmetic is fp32 (expect ~1e-5 relative to an fp64 evaluation).
 * Supported: d = 64 or 128, G <= 64, and for both K and V of the layer n = 64 or 256 with
 * 8-bit linear or 4-bit log-space norms (TVQ_ERR_UNSUPPORTED otherwise).  Launches two
 * kernels on `stream`. */
tvq_status tvq_attention_workspace(const tvq_codec* c, int64_t batch, int32_t num_q_heads,
                                   int64_t t_end, int64_t* bytes);
tvq_status tvq_attention_decode(const tvq_codec* c, const void* cache, const tvq_layout* lay,
                                int32_t layer, int64_t t_end, int32_t num_q_heads, float scale,
                                tvq_dtype q_dtype, const void* q, tvq_dtype o_dtype, void* o,
                                void* workspace, int64_t workspace_bytes, void* stream);

/* Bytes of the device scratch that tvq_attention_decode_noalloc uses in place of a workspace:
 * one static array per GPU, held from the library's first use of that GPU until the process
 * ends (16 MiB; the long-context shape of 16 sequences x 32 query heads x 32K tokens at d = 128
 * needs 8.5 MB). */
#define TVQ_ATTENTION_SCRATCH_BYTES (16 * 1024 * 1024)

/* tvq_attention_decode without the workspace argument, for callers that cannot allocate
 * device memory (code under graph capture, serving loops that forbid allocation): the
 * per-chunk partials go to the library's static scratch on the codec's device.  Allocates
 * nothing and calls no allocating routine; arguments, results and launches are those of
 * tvq_attention_decode.  TVQ_ERR_SCRATCH, with nothing launched, when the call's partials
 * (the chunks planned for this layer's formats) exceed TVQ_ATTENTION_SCRATCH_BYTES; TVQ_ERR_HIP when the scratch's
 * device address could not be obtained at tvq_create.  Every call on one GPU shares that
 * scratch: calls that overlap in time on one GPU (concurrent streams, or host threads each
 * launching) race on it and must be ordered by the caller.  The scratch needs no clearing:
 * each call writes every partial it reads. */
tvq_status tvq_attention_decode_noalloc(const tvq_codec* c, const void* cache,
                                        const tvq_layout* lay, int32_t layer, int64_t t_end,
                                        int32_t num_q_heads, float scale, tvq_dtype q_dtype,
                                        const void* q, tvq_dtype o_dtype, void* o, void* stream);

/* ---- paged caches (serving) ----
 * A paged pool holds fixed-size blocks of cache slots shared by many sequences.  Its byte
 * layout is that of tvq_cache_layout(c, n_blocks, block_tokens): block j plays the part of
 * "sequence" j, so the record of (block j, head h, row r) sits at ((j*H + h)*block_tokens + r)
 * in every plane.  block_tokens is a power of two in [32, 65536].  A block table, device int32
 * [B][max_blocks] with max_blocks * block_tokens < 2^31, maps position t of sequence b to
 * pool block table[b][t / block_tokens], row t % block_tokens.  Per-sequence positions and
 * lengths are device data too, so one call serves every step of a decode loop and can be
 * captured in a HIP graph and replayed while the caller advances them on the device.
 * Positions past a sequence's table row, or whose entry holds no pool block (< 0 or
 * >= n_blocks), are skipped by encode and decode to zeros.  Attention reads positions below
 * each context, clipped to max_blocks * block_tokens; they must lie in blocks the table
 * holds: an entry holding no pool block is read as pool block 0 (memory-safe, meaningless
 * values). */

/* Encode (as tvq_encode) in->tokens tokens of each of the in->batch sequences into a paged
 * pool: token t of sequence b goes to position positions[b] + t through the block table
 * (positions: device int32 [in->batch]; a negative position writes nothing).  One or two
 * kernel launches (as tvq_encode); with in->tokens == 1 this is the per-step append. */
tvq_status tvq_encode_paged(const tvq_codec* c, tvq_dtype in_dtype, const void* k, const void* v,
                            const tvq_tensor_desc* in, const int32_t* positions,
                            const int32_t* block_table, int32_t max_blocks, void* pool,
                            const tvq_layout* pool_layout, void* stream);

/* Decode (as tvq_decode) positions [t_begin, t_end) of the out->batch sequences of a paged
 * pool into k_out / v_out (out->tokens == t_end - t_begin, t_end <= max_blocks *
 * block_tokens).  Launches as tvq_decode: up to two kernels on `stream` (one for the layers
 * whose formats have a dedicated kernel, one for the rest), twice over for a range of at least
 * 2^19 vectors per kind that starts on a multiple of the tile's token count and whose token
 * count is not one; an empty range launches nothing. */
tvq_status tvq_decode_paged(const tvq_codec* c, const void* pool, const tvq_layout* pool_layout,
                            const int32_t* block_table, int32_t max_blocks, int64_t t_begin,
                            int64_t t_end, tvq_dtype out_dtype, void* k_out, void* v_out,
                            const tvq_tensor_desc* out, void* stream);

/* Attention (as tvq_attention_decode) of `batch` sequences over a paged pool: sequence b
 * attends its positions [0, min(ctx_lens[b], max_ctx)) (ctx_lens: device int32 [batch];
 * <= 0 gives a zero output).  max_ctx (host, 1 .. max_blocks * block_tokens) bounds every
 * context and fixes the launch shape, so the call can be replayed as the lengths grow.  The
 * workspace is at least tvq_attention_paged_workspace(c, batch, num_q_heads, max_ctx,
 * block_tokens) bytes.  Two kernel launches on `stream`. */
tvq_status tvq_attention_paged_workspace(const tvq_codec* c, int64_t batch, int32_t num_q_heads,
                                         int64_t max_ctx, int64_t block_tokens, int64_t* bytes);
tvq_status tvq_attention_paged(const tvq_codec* c, const void* pool, const tvq_layout* pool_layout,
                               const int32_t* block_table, int32_t max_blocks,
                               const int32_t* ctx_lens, int64_t max_ctx, int64_t batch,
                               int32_t layer, int32_t num_q_heads, float scale, tvq_dtype q_dtype,
                               const void* q, tvq_dtype o_dtype, void* o, void* workspace,
                               int64_t workspace_bytes, void* stream);

/* Bits per element of the codec, averaged over layers and over K and V.
 * accounting 0: the paper's -- eq. (1) angle bits (log2 n)/2 (fractional for non-power-of-
 *               two n) plus, per eq. (3), b_norm/2 + 64/d for quantized norms or 16 for
 *               fp32 norms (section 3.1 "Rate accounting");
 * accounting 1: actual storage of the layout above (ceil(log2 n) bits per angle code).
 * Returns a negative value for a NULL codec or an unknown accounting. */
double tvq_bits_per_element(const tvq_codec* c, int accounting);

/* Static description of a status code. */
const char* tvq_status_string(tvq_status s);

/* ---- host-only helpers (no GPU needed) ---- */

/* The sign row of `layer` drawn from `seed`: out[i] = +1 iff the top bit of
 * SplitMix64 output i+1 of the stream keyed by mix(seed ^ (layer+1)*0xD1B54A32D192ED03)
 * is 0 (mix = the SplitMix64 finalizer; stream output j = mix(key + j*0x9E3779B97F4A7C15)). */
tvq_status tvq_make_signs(uint64_t seed, int32_t layer, int32_t head_dim, int8_t* out);

/* The reconstruction lookup table of an n-bin codebook (section 3.1): cos_out[k], sin_out[k]
 * = fp32 roundings of cos(2 pi k/n), sin(2 pi k/n), exact at multiples of pi/4. */
tvq_status tvq_make_trig_table(int32_t n, float* cos_out, float* sin_out);

/* The table the decode kernels read for an n-bin codebook at head dimension d: the same fp64
 * values divided by sqrt(d) (the normalization of H, section 2) and rounded once to fp32,
 * cos_out[k] = RN32(cos(2 pi k/n) / sqrt(d)), sin_out[k] likewise.  Host-only. */
tvq_status tvq_make_decode_table(int32_t n, int32_t head_dim, float* cos_out, float* sin_out);

/* The angle bins the encode kernels read for an n-bin codebook, n a power of two in
 * [16, 256] (Algorithm 1: k = round(n theta / 2 pi) mod n, round = floor(u + 1/2)).  A pair
 * (a, b) is placed by p' = sign(a) b / (|a| + |b|) in [-1, 1]: for each sign of a (h = 0 for a
 * sign bit of 0, h = 1 for 1) p' moves monotonically over half a turn of angles.  With
 * K = n - 3 equal cells of [-1, 1], entry h n + i covers: i = 0, p' < -1 (a rounding
 * overshoot); i = 1 .. K, cell i - 1, p' in [-1 + 2 (i - 1) / K, -1 + 2 i / K); i = K + 1,
 * p' >= 1; i > K + 1 repeats entry K + 1.  code_out[h n + i] is the code at the entry's lowest
 * p'; bound_out[h n + i] the fp32 rounding of the p' of the one bin boundary inside the cell,
 * from which the code is one more (mod n), or 3 where the cell holds none.  Both arrays hold
 * 2 n entries.  Host-only; TVQ_ERR_INVALID_ARG for other n or null pointers. */
tvq_status tvq_make_angle_bins(int32_t n, uint32_t* code_out, float* bound_out);

/* The constants of the encode kernels' fp32 arithmetic, so that a host program can run the
 * same steps (Algorithm 1, the angle quantizer; section 3.3, eq. (2) and its log-space variant):
 *   poly_out[6]   the coefficients of atan(t)/(2 pi) = t * p(t^2), t in [0, 1], from the
 *                 highest power of t^2 down, that the evaluated angle path uses;
 *   spread_out[2] the range [lo, hi) of bits(s2_max) - bits(s2_min) (the bit patterns of a
 *                 vector's largest and smallest squared pair norm) inside which a vector's norm
 *                 codes come from fp32 formulas; a tile holding any other vector takes its
 *                 norm codes from fp64.
 * Host-only.  TVQ_ERR_INVALID_ARG for null pointers. */
tvq_status tvq_encode_constants(float* poly_out, uint32_t* spread_out);

/* Layout of a configuration without creating a codec (same result as tvq_cache_layout). */
tvq_status tvq_layout_for_config(const tvq_config* cfg, int64_t batch, int64_t capacity_tokens,
                                 tvq_layout* out);

/* tvq_bits_per_element for a configuration without creating a codec.  Returns a negative
 * value for an invalid configuration or accounting. */
double tvq_bits_per_element_config(const tvq_config* cfg, int accounting);

/* TVQ_ABI_VERSION of the built library. */
int32_t tvq_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* TVQ_H */
