/*
 * fdkv.h - C ABI of the FreqDepthKV compressed-KV path on AMD MI355X (gfx950).
 *
 * FreqDepthKV (Section 3 of the paper) compresses a decoder's KV cache along
 * depth.  Adjacent layers form blocks of B = 2 or 4; an orthonormal DCT along
 * the layer axis (Eq. 1) splits each block into a low-frequency coefficient
 * stored once for the block and high-frequency coefficients kept only
 * sparsely (Eq. 3).  An online probe measures, per (block, KV head), how much
 * each candidate reconstruction moves the attention logits of probe queries
 * (Eq. 2) and routes the head to one of three modes; decode attention then
 * rebuilds K/V on the fly inside a fused softmax(q K^T) V.
 *
 * Conventions shared by every entry point:
 *
 *  - `dims.schedule` cuts the layers into blocks (fdkv_blocks lists them):
 *    all pairs, all blocks of four, or the paper's default setting (Section
 *    4): pairs for the first four and the last four layers, blocks of four
 *    between.  A block of B layers starts at a multiple of B.  A "unit" is a
 *    (block, KV head); unit arrays are [n_blocks][Hkv].
 *  - Every block stores the mean of its layers, M (the per-layer image of
 *    the low-frequency DCT-II coefficient), as its shared part.
 *  - Pairs (layers l, l+1): D = (x[l] - x[l+1]) / 2; layer l rebuilds M + D,
 *    layer l+1 rebuilds M - D.  The residual of a token keeps the `topk`
 *    channels of largest |fl32(x[l] - x[l+1])| (ties to the lower channel),
 *    as uint8 channel indices in ascending order plus D at those channels.
 *  - Blocks of four: Z_j = sum_n F_4[j][n] x[l+n], j = 1..3, with F_4 the
 *    orthonormal DCT-II(4), F_4[j][n] = cos(pi (2n+1) j / 8) / sqrt(2).  The
 *    residual of a token keeps the `topk` largest of its 3d coefficients
 *    |Z_j[c]|, ranked as fp32 evaluates the butterfly
 *      Z_1 = a (x0 - x3) + b (x1 - x2),  Z_2 = ((x0 + x3) - (x1 + x2)) / 2,
 *      Z_3 = b (x0 - x3) - a (x1 - x2),  a = F_4[1][0], b = F_4[1][1]
 *    (each product and sum rounded), ties to the lower code; it stores the
 *    uint16 codes 4c + j in ascending order plus Z_j[c].  Layer l+p rebuilds
 *    M plus F_4[j][p] Z_j[c] at channel c for each kept code.
 *  - K and V choose their residual entries independently.
 *  - dims.residual = FDKV_RES_TOKENS switches residual heads to the
 *    paper's token-level set (Section 3, after Eq. 2): every high-frequency
 *    coefficient (pairs: D; fours: Z_1..Z_3) of the n = ceil(r T) tokens,
 *    r = res_ppm / 10^6 (or, with dims.n_rates > 0, the unit's own fraction
 *    r_j = rates_ppm[j] / 10^6, j given by its mode byte), with the largest score
 *      s_t = max over the probe rows q of every layer of the block and every
 *            query head of the group of |q . (K_t - K^S_t)|,
 *    K - K^S computed in fp32 on the stored inputs and rounded to bf16 (pairs:
 *    (x0 - x1) / 2 up to sign; fours: x_l - ((x0 + x3) + (x1 + x2)) / 4);
 *    ties go to the lower token.  fdkv_probe writes the scores and
 *    fdkv_compress selects from them (K and V share the set).
 *  - Query head g reads KV head g / (n_q_heads / n_kv_heads).
 *  - K, V, queries, the cache and attention outputs use one element type,
 *    `dims.dtype` (fp32 or bf16); all arithmetic is fp32.
 *  - Device pointers are caller-owned device memory, 16-byte aligned.  The
 *    library allocates nothing, keeps no state between calls and launches
 *    work asynchronously on the caller's stream (`stream` is a hipStream_t;
 *    NULL means the null stream).  Host-side validation happens before any
 *    HIP call, so an invalid argument never touches the device.
 *  - Kernel launch failures return FDKV_E_HIP; faults inside a kernel
 *    surface at the caller's next synchronisation.  Inputs must be finite.
 *
 * Compressed cache layout (one device buffer).  It is a sequence of
 * segments, one per (sequence, block, KV head) in row-major order, each
 * starting at the offset fdkv_layout() returns.  A segment is a list of
 * planes, each padded to a multiple of 256 bytes; e = bytes of an input
 * element, c = bytes of a stored coefficient, i = 1 (pairs) or 2 (blocks of
 * four) bytes of a residual index:
 *    SHARED   : MK[T][d] (c), MV[T][d] (c)
 *    RESIDUAL : MK, MV, IK[T][k] (i), VK[T][k] (c), IV[T][k] (i), VV[T][k] (c)
 *    EXACT    : K of the B layers [T][d] (e) in order, then V of the B layers
 * With FDKV_RES_TOKENS a residual segment is instead
 *    MK, MV, MASK[ceil(T/32)] (u32, bit t%32 of word t/32: token t is in the
 *    set), COUNT[ceil(T/128) + 1] (u32, set tokens before each 128-token
 *    chunk, then n), HK[n][B-1][d] (c), HV[n][B-1][d] (c)  (set tokens ascending)
 * FP8 shared planes (MK, MV with c = 1) are not row-major: they fill whole
 * 1 KB blocks of R = 1024/d rows, and the 8 channels 8p .. 8p+7 of row t sit
 * at byte 1024 (t / R) + 16 ((t % (R/2)) d/8 + p) + 8 ((t % R) / (R/2)), so
 * rows t and t + R/2 of a block share each 16-byte slot.  Every other plane
 * is row-major.
 */
#ifndef FDKV_H
#define FDKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FDKV_OK = 0,
  FDKV_E_INVALID_ARG = -1, /* null/misaligned pointer, bad size or shape */
  FDKV_E_UNSUPPORTED = -2, /* valid but not compiled: head_dim not 64/128, group not 1/2/4/8 */
  FDKV_E_WORKSPACE = -3,   /* workspace smaller than the *_workspace query returned */
  FDKV_E_BUDGET = -4,      /* byte budget below the all-shared footprint */
  FDKV_E_HIP = -5          /* a HIP runtime call failed (see fdkv_last_error) */
} fdkv_status;

/* Head modes, in increasing memory cost; ties in routing go to the lower value.
 * A unit's mode byte holds the mode in bits 0-1; with token-level sets whose
 * fraction is routed per unit (dims.n_rates > 0) a residual unit's byte also
 * holds, in bits 2-4, the index j of its fraction rates_ppm[j].  Every other
 * byte is invalid. */
typedef enum { FDKV_SHARED = 0, FDKV_RESIDUAL = 1, FDKV_EXACT = 2 } fdkv_mode;

/*
 * Cache types.  FDKV_F32 / FDKV_BF16: inputs, queries, outputs and every cache
 * plane in that type.  FDKV_BF16_E4M3: bf16 inputs, queries, outputs and exact
 * heads, with the shared planes and residual values of shared / residual heads
 * stored as OCP FP8 E4M3 (the quantised coefficients Section 3 allows), each
 * rounded once to nearest-even from its fp32 value and saturated at +-448.
 */
typedef enum { FDKV_F32 = 0, FDKV_BF16 = 1, FDKV_BF16_E4M3 = 2 } fdkv_dtype;

/*
 * Block schedules.  PAIRS: every block two layers (L even).  MIXED: two
 * pairs, blocks of four, two pairs (L >= 8, L - 8 a multiple of 4), the
 * default of Section 4.  QUADS: every block four layers (L a multiple of 4).
 */
typedef enum { FDKV_SCHED_PAIRS = 0, FDKV_SCHED_MIXED = 1, FDKV_SCHED_QUADS = 2 } fdkv_schedule;

/* Residual kinds: per-token top-k channel entries, or the token-level set. */
typedef enum { FDKV_RES_CHANNELS = 0, FDKV_RES_TOKENS = 1 } fdkv_residual;

typedef struct {
  int32_t n_layers;   /* L, 2..128, fitting the schedule */
  int32_t n_kv_heads; /* Hkv >= 1 */
  int32_t n_q_heads;  /* Hq, a multiple of Hkv; Hq / Hkv in {1, 2, 4, 8} */
  int32_t head_dim;   /* d in {64, 128} */
  int32_t topk;       /* k residual channels per token, 0 <= k <= d */
  int32_t dtype;      /* fdkv_dtype */
  int32_t schedule;   /* fdkv_schedule */
  int32_t residual;   /* fdkv_residual */
  int32_t res_ppm;    /* FDKV_RES_TOKENS: the set's fraction of tokens, 0..10^6 parts per million */
  int32_t n_rates;    /* FDKV_RES_TOKENS: 0, every residual head keeps res_ppm of its tokens; 1..8, each
                         residual head keeps one of rates_ppm[0..n_rates), chosen by fdkv_route */
  int32_t rates_ppm[8]; /* the candidate fractions, strictly increasing, 0..10^6 */
} fdkv_dims;

/* Message for a status code (static storage). */
const char* fdkv_status_string(int32_t status);

/* Text of the last failure in the calling thread that carries a message (every
 * FDKV_E_HIP, and FDKV_E_WORKSPACE from fdkv_decode_attn_static); "" if none. */
const char* fdkv_last_error(void);

/*
 * fdkv_blocks - host only.  The blocks of dims.schedule, in layer order.
 *   n_blocks     host  out: number of blocks (at most L/2)
 *   first_layer  host [n_blocks] or NULL  out: first layer of each block
 *   block_size   host [n_blocks] or NULL  out: 2 or 4
 */
fdkv_status fdkv_blocks(const fdkv_dims* dims, int32_t* n_blocks, int32_t* first_layer, int32_t* block_size);

/*
 * fdkv_layout - host only.  Byte layout of a compressed cache (Eq. 3 storage).
 *   seq_lens     host [batch]                     tokens per sequence, >= 0
 *   modes        host [batch][n_blocks][Hkv]           fdkv_mode per unit
 *   seg_offsets  host [batch][n_blocks][Hkv] or NULL   out: segment byte offsets
 *   total_bytes  host                                  out: buffer size needed
 * Segments follow each other in (sequence, block, head) order; all offsets
 * are multiples of 256.
 */
fdkv_status fdkv_layout(const fdkv_dims* dims, int32_t batch, const int32_t* seq_lens,
                        const uint8_t* modes, uint64_t* seg_offsets, uint64_t* total_bytes);

/*
 * fdkv_route - host only.  Mode choice of Eq. (3), m = argmin E_m + lambda * Omega(m)
 * with Eq. (2)'s loss, and the budget rule that raises lambda until the cache
 * fits (end of Section 3).  With routed fractions (dims.n_rates = J > 0) the
 * residual mode at each fraction r_j is a candidate of its own (loss E_R(r_j),
 * Omega of its bytes), so each residual unit also gets its fraction (Section
 * 3: r_{b,h} chosen by the routing loss budget).
 *   seq_len      tokens of the sequence (for the footprint)
 *   errors       host [n_blocks][Hkv][2]   E_shared, E_residual per unit
 *                                          (E_exact = 0), as written by fdkv_probe;
 *                with routed fractions [n_blocks][Hkv][1 + J]: E_shared, E_residual(r_0..r_{J-1})
 *   lambda       penalty used when budget_bytes == 0
 *   budget_bytes 0: route with `lambda`.  Otherwise: the smallest lambda among
 *                0, the per-unit breakpoints (E_i - E_j)/(Omega_j - Omega_i)
 *                and +inf whose fdkv_layout footprint is <= budget_bytes.
 *   modes_out    host [n_blocks][Hkv]   out: mode bytes
 *   lambda_out   host, may be NULL out: lambda used (+inf when infeasible)
 * Omega(m) = bytes per token of mode m / bytes per token of EXACT, for the
 * unit's block size.  Ties go to the cheaper candidate; two candidates are
 * compared through their breakpoint, so at a lambda equal to it the tie is exact.  Returns FDKV_E_BUDGET (modes all SHARED) when even
 * all-shared exceeds the budget.
 */
fdkv_status fdkv_route(const fdkv_dims* dims, int32_t seq_len, const float* errors, double lambda,
                       uint64_t budget_bytes, uint8_t* modes_out, double* lambda_out);

/* Device workspace bytes fdkv_probe needs for this shape. */
fdkv_status fdkv_probe_workspace(const fdkv_dims* dims, int32_t seq_len, int32_t n_probe, size_t* bytes);

/* Bytes of the K selection buffer that fdkv_probe may fill and fdkv_compress
 * may read: the per-token residual selection of K of every unit (top-k
 * channels of a pair, top-k coefficients of a block of four), in an internal
 * layout of d * elem_bytes / 16 slots per unit and token, a slot being 1 byte,
 * or 4 when the schedule has blocks of four. */
fdkv_status fdkv_selection_bytes(const fdkv_dims* dims, int32_t seq_len, size_t* bytes);

/*
 * fdkv_probe - device.  Routing loss of Eq. (2) for every (block, KV head):
 *   E_m[b,h] = 1/(B G P) * sum over the B layers l of the block, query heads g
 *              of KV head h, probe rows p, tokens t of
 *              ((q_{l,g,p} . (K^(m)_{l,h,t} - K_{l,h,t})) / sqrt(d))^2
 * for m = SHARED (K^ = M) and m = RESIDUAL (K^ = M plus the token's kept
 * residual entries).  Logits are compared raw, over all T keys, for keys only.
 *   k_layers   host array of L device pointers, layer l holds K_l [Hkv][T][d]
 *   qp_layers  host array of L device pointers, layer l holds Q_l [Hq][P][d]
 *   n_probe    P >= 1 probe rows per query head
 *   errors_out device float [n_blocks][Hkv][2], or [n_blocks][Hkv][1 + J] with J = dims.n_rates > 0
 *              routed fractions (E_residual at each)
 *   token_scores_out  FDKV_RES_TOKENS: device float [n_blocks][Hkv][T], out: s_t
 *                     (the residual loss then keeps the top ceil(r T) tokens); else unused
 *   ws         device workspace of >= fdkv_probe_workspace() bytes
 *   k_select_out  device, NULL or fdkv_selection_bytes() bytes (4-byte aligned), out:
 *              the per-token residual selection of K that the residual loss uses
 *              (Eq. 3), for fdkv_compress of the same keys to reuse; unused with
 *              FDKV_RES_TOKENS
 * T * d * elem_bytes and P * G * d * elem_bytes must stay below 2^31
 * (FDKV_E_UNSUPPORTED otherwise: planes are addressed with 32-bit offsets).
 */
fdkv_status fdkv_probe(const fdkv_dims* dims, int32_t seq_len, const void* const* k_layers,
                       const void* const* qp_layers, int32_t n_probe, float* errors_out,
                       float* token_scores_out, void* ws, size_t ws_bytes, uint8_t* k_select_out,
                       void* stream);

/*
 * fdkv_compress - device.  Writes one sequence's segments of the compressed
 * cache (Eq. 1 factorization, Eq. 3 storage) for the given modes.
 *   k_layers, v_layers  host arrays of L device pointers, [Hkv][T][d] each
 *   modes        device [n_blocks][Hkv]
 *   seg_offsets  device [n_blocks][Hkv], from fdkv_layout (256-byte multiples)
 *   token_scores FDKV_RES_TOKENS: device float [n_blocks][Hkv][T] from fdkv_probe; else unused
 *   k_select     device, NULL (residual units select their K entries in the pass)
 *                or the buffer fdkv_probe filled for these k_layers and seq_len
 *                (residual units then take their K entries' positions from it: the
 *                same selection, without ranking again); unused with FDKV_RES_TOKENS
 *   cache        device buffer the offsets index into
 */
fdkv_status fdkv_compress(const fdkv_dims* dims, int32_t seq_len, const void* const* k_layers,
                          const void* const* v_layers, const uint8_t* modes,
                          const uint64_t* seg_offsets, const float* token_scores, const uint8_t* k_select,
                          void* cache, void* stream);

/* Device workspace bytes fdkv_decode_attn needs for this batch shape. */
fdkv_status fdkv_decode_workspace(const fdkv_dims* dims, int32_t batch, int32_t max_seq_len, size_t* bytes);

/*
 * fdkv_decode_attn - device.  One decode step of one layer over the
 * compressed cache, with the reconstruction of Eq. (3) fused into attention
 * (Section 3, after Eq. 3): o = softmax(q K~^T * sm_scale) V~ over the T_i
 * cached tokens of each sequence, K~/V~ rebuilt per head mode.
 *   seq_lens     device int32 [batch], 0 <= T_i <= max_seq_len (T_i = 0 gives o = 0)
 *   max_seq_len  host, sizes the launch; max_seq_len * d * elem_bytes < 2^31
 *                (FDKV_E_UNSUPPORTED otherwise: planes are addressed with 32-bit offsets)
 *   modes        device [batch][n_blocks][Hkv], 4-byte aligned and allocated to a
 *                multiple of 4 bytes (read in aligned 4-byte words; the padding
 *                bytes are ignored)
 *   seg_offsets  device [batch][n_blocks][Hkv]
 *                A unit whose mode is above FDKV_EXACT or whose offset is not a
 *                multiple of 256 is not read: the outputs of its query heads
 *                come out NaN, so a corrupt mode table cannot pass unnoticed.
 *   layer        0 <= layer < L
 *   q            device [batch][Hq][d]
 *   out          device [batch][Hq][d]
 *   sm_scale     logit scale (the paper uses 1/sqrt(d))
 *   ws           device workspace of >= fdkv_decode_workspace() bytes
 */
fdkv_status fdkv_decode_attn(const fdkv_dims* dims, int32_t batch, const int32_t* seq_lens,
                             int32_t max_seq_len, const uint8_t* modes, const uint64_t* seg_offsets,
                             const void* cache, int32_t layer, const void* q, void* out,
                             float sm_scale, void* ws, size_t ws_bytes, void* stream);

/*
 * fdkv_decode_partial / fdkv_decode_combine - device.  The two phases of
 * fdkv_decode_attn, for callers that merge partial attention results
 * themselves: a sequence split over several devices runs the partial phase
 * on each device's tokens, gathers the records and combines them once (the
 * log-sum-exp merge is associative and order-free).
 * fdkv_decode_partial takes the arguments of fdkv_decode_attn minus `out`
 * and writes the split-K records into ws: for every (sequence, KV head,
 * 512-token chunk) slot and every query head g of the KV head's group, d + 4
 * floats
 *   acc[0..d) = sum_t 2^(z_t - m) V~_t,  m = a reference max of z_t,
 *   l         = sum_t 2^(z_t - m),      then 2 floats of padding,
 * with z_t = (q . K~_t) sm_scale log2(e) over the chunk's tokens; records are
 * laid out [batch][Hkv][n_chunks][G][d + 4], n_chunks = ceil(max_seq_len / 512),
 * and a slot with no tokens holds m = -inf, l = 0, acc = 0.
 * fdkv_decode_combine merges, per (sequence, query head), the n_chunks records
 * of ws (the same layout, any n_chunks >= 1):
 *   o = sum_i 2^(m_i - M) acc_i / sum_i 2^(m_i - M) l_i,  M = max_i m_i,
 * and writes o in the cache type (o = 0 when no slot holds a token).
 *   ws_bytes >= batch x Hkv x n_chunks x G x (d + 4) x 4 (FDKV_E_WORKSPACE otherwise)
 */
fdkv_status fdkv_decode_partial(const fdkv_dims* dims, int32_t batch, const int32_t* seq_lens, int32_t max_seq_len,
                                const uint8_t* modes, const uint64_t* seg_offsets, const void* cache, int32_t layer,
                                const void* q, float sm_scale, void* ws, size_t ws_bytes, void* stream);
fdkv_status fdkv_decode_combine(const fdkv_dims* dims, int32_t batch, int32_t n_chunks, void* out, const void* ws,
                                size_t ws_bytes, void* stream);

/*
 * fdkv_decode_attn_static - device.  fdkv_decode_attn for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same computation and arguments
 * without the workspace.  Its split-K records live in a static device array
 * of the library, fdkv_decode_static_scratch_bytes() bytes (16 MiB), one per
 * GPU, held until the process ends; the call itself allocates nothing.
 *   Returns FDKV_E_WORKSPACE (message in fdkv_last_error) when the call needs
 *   more than that, i.e. fdkv_decode_workspace(dims, batch, max_seq_len) >
 *   fdkv_decode_static_scratch_bytes(): batch x Hkv x ceil(max_seq_len / 512) x
 *   G x (d + 4) x 4 bytes (the 8B shape at 32k tokens needs 1 MiB, the 70B shape
 *   at 131k tokens 8.3 MiB).
 * Every call on one GPU shares that GPU's array (the current device's), which
 * keeps the last call's records: calls that overlap on one GPU (on different
 * streams, or from different host threads without ordering) race and must
 * not be issued.  Nothing in the array needs clearing between calls: each
 * call writes every record it reads.
 */
size_t fdkv_decode_static_scratch_bytes(void);
fdkv_status fdkv_decode_attn_static(const fdkv_dims* dims, int32_t batch, const int32_t* seq_lens,
                                    int32_t max_seq_len, const uint8_t* modes, const uint64_t* seg_offsets,
                                    const void* cache, int32_t layer, const void* q, void* out, float sm_scale,
                                    void* stream);

/*
 * Generation (the end of Section 3's method): one routing after prefill
 * serves the whole decode, optionally re-decided at a fixed period of
 * generated tokens.  Here a cache is a list of compressed spans
 * (prefill is span 0; each refresh compresses the tokens generated since
 * the last one into a new span, routed by fdkv_probe / fdkv_route on those
 * tokens' own keys) followed by an exact tail that holds the tokens not yet
 * compressed.  Every span is an ordinary compressed cache (fdkv_layout,
 * fdkv_compress) of its own tokens; decode attends over all spans and the
 * tail in one softmax.
 */
typedef struct {
  const int32_t* seq_lens;      /* device [batch]: tokens of each sequence in this span */
  int32_t max_seq_len;          /* host: the largest entry of seq_lens (sizes the launch) */
  const uint8_t* modes;         /* device [batch][n_blocks][Hkv], 4-byte aligned, padded to 4 bytes */
  const uint64_t* seg_offsets;  /* device [batch][n_blocks][Hkv] */
  const void* cache;            /* device, 256-byte aligned */
} fdkv_span;

typedef struct {
  const int32_t* lens;          /* device [batch]: rows held by each sequence's tail, 0..cap */
  int32_t cap;                  /* host: rows per (sequence, KV head) */
  const void* k;                /* device [batch][Hkv][cap][d] of the decoded layer */
  const void* v;
} fdkv_tail;

/*
 * fdkv_append - device.  Writes one layer's new K and V rows into the exact
 * tail: row pos[s] of every (sequence s, KV head).
 *   pos            device int32 [batch]; a sequence whose pos is outside
 *                  [0, cap) is skipped (nothing written)
 *   cap            rows per (sequence, KV head) of the tail
 *   k_new, v_new   device [batch][Hkv][d] (the layer's new token)
 *   tail_k, tail_v device [batch][Hkv][cap][d] (the layer's tail)
 */
fdkv_status fdkv_append(const fdkv_dims* dims, int32_t batch, const int32_t* pos, int32_t cap,
                        const void* k_new, const void* v_new, void* tail_k, void* tail_v, void* stream);

/* Device workspace bytes fdkv_decode_spans needs: max_seq_lens host [n_spans],
 * tail_cap the tail's cap, or -1 for no tail.  At most 16 parts (spans + tail). */
fdkv_status fdkv_decode_spans_workspace(const fdkv_dims* dims, int32_t batch, int32_t n_spans,
                                        const int32_t* max_seq_lens, int32_t tail_cap, size_t* bytes);

/*
 * fdkv_decode_spans - device.  One decode step of one layer over n_spans
 * compressed spans and an optional exact tail (NULL: none):
 * o = softmax(q K~^T * sm_scale) V~ over every span's reconstructed tokens
 * and the tail's rows, as fdkv_decode_attn computes it for one span.  A
 * sequence with no token in any part gets o = 0.  spans is a host array of
 * n_spans descriptors; the same limits as fdkv_decode_attn apply to each
 * span, and cap * d * elem_bytes < 2^31 to the tail.
 */
fdkv_status fdkv_decode_spans(const fdkv_dims* dims, int32_t batch, int32_t n_spans, const fdkv_span* spans,
                              const fdkv_tail* tail, int32_t layer, const void* q, void* out, float sm_scale,
                              void* ws, size_t ws_bytes, void* stream);

/*
 * fdkv_check_conversions - diagnostic, synchronous on `stream`.  Runs the
 * device's number encoders over every fp32 bit pattern except NaN and
 * counts where they differ from their integer definitions (0 expected):
 *   mismatches[0]  the E4M3 encoder of the compress kernels (the conversion
 *                  instruction on inputs clamped to +-448) against round to
 *                  nearest even with saturation at 448 (Section 3's
 *                  quantised coefficients, OCP E4M3)
 *   mismatches[1]  the bf16 pair conversion against round to nearest even
 *                  on the bit pattern
 *   mismatches     host uint64 [2], out
 * Allocates and frees 16 bytes of device memory; FDKV_E_HIP on a runtime error.
 */
fdkv_status fdkv_check_conversions(uint64_t* mismatches, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FDKV_H */
