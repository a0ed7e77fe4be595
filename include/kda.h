/*
 * kda.h — C ABI of libkda: the Kimi Delta Attention (KDA) recurrence with a
 * decay-aware mixed-precision recurrent state, for AMD Instinct MI355X (gfx950).
 *
 * Method: "Low-Bit Recurrent States in Hybrid Language Models"
 * (arxiv 2609.30950).  Per head, the state S (d_k x d_v, rows = key channels)
 * follows the gated delta rule (Sec. 2, eq. rule) with the KDA choice of erase
 * and write vectors:
 *
 *     S_t = (I - beta_t k_t k_t^T) diag(exp(-s_t)) S_{t-1} + beta_t k_t v_t^T,
 *     o_t = S_t^T q_t,
 *
 * and is written back every C tokens as Deq(Q(S)) (Sec. 2, Accumulated
 * readout error; Sec. 5, Protocol): outputs are read before quantisation and no
 * unquantised residual is kept.  Q is the paper's quantiser (Sec. 3):
 * per-row widths from the high-rate allocation rule (eq. alloc) on weights
 * c_i = Gamma_i * R~_i^2 (eq. weight), symmetric levels with a clip factor
 * fitted over 16 values and stored as an FP16 scale, variable-width rows
 * addressed by prefix sums of widths, and log-uniform codes of the decay rate.
 *
 * Conventions for every entry point
 * ---------------------------------
 * - All array arguments are DEVICE pointers (HIP device memory) unless stated;
 *   the config is a host pointer.  Arrays are dense, C-contiguous, in the
 *   layout given per argument; the caller owns every buffer.
 * - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *   Every call only enqueues work on `stream`: it never synchronises, never
 *   allocates device memory and never prints.
 * - Arguments are validated before anything is enqueued; on any error nothing
 *   is launched and a kda_status other than KDA_OK is returned.  Empty
 *   requests are errors: B or H below 1 give KDA_ERR_SHAPE, a token count T,
 *   window W or write-back interval C below 1 gives KDA_ERR_ARG.  A failed
 *   kernel launch returns KDA_ERR_HIP.  NaN/Inf in inputs are not checked.
 * - Records: one fixed-size slot of kda_record_bytes() per (sequence, head),
 *   slots ordered [B][H].  A zero-filled slot is the zero state (fresh EMA).
 *   kda_step / kda_prefill update records in place.
 * - Records, workspace and state arrays must be 16-byte aligned (device
 *   allocations are); misaligned pointers give KDA_ERR_ARG.
 * - Workspace: kda_workspace_bytes() bytes, used as scratch by one call at a
 *   time (per-row weights, widths, rate codes, and between the passes of a
 *   write-back either the token's vectors a, g, w (decode, d_k <= 128: the
 *   requantisation rebuilds the state from the record) or the float32 state
 *   (prefill, d_k = 256)).  Concurrent calls must not share one.
 */
#ifndef KDA_H_
#define KDA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  KDA_OK = 0,
  KDA_ERR_ARG = 1,          /* bad pointer, size or numeric parameter        */
  KDA_ERR_SHAPE = 2,        /* unsupported or inconsistent shape             */
  KDA_ERR_UNSUPPORTED = 3,  /* valid request the library does not implement   */
  KDA_ERR_WORKSPACE = 4,    /* workspace pointer missing                     */
  KDA_ERR_HIP = 5           /* a HIP runtime call or kernel launch failed    */
} kda_status;

enum { KDA_SCOPE_SEQUENCE = 0, KDA_SCOPE_HEAD = 1 };

/* Problem and quantiser configuration (host memory, plain old data). */
/* Allocation-key variants (Sec. 5, Table ablate).  Gamma^ = 1/expm1(2 (s^ +
 * r)) (eq. weight), R~ the normalised range, R the raw row maximum, rates
 * clamped below at 1e-12; given weights (`gamma` arguments) replace the
 * factor in front of the range term. */
typedef enum {
  KDA_WEIGHT_EMA = 0,           /* Gamma^ R~^2 (the paper's method)            */
  KDA_WEIGHT_RANGE = 1,         /* R^2 (range alone)                           */
  KDA_WEIGHT_GAMMA_RANGE = 2,   /* Gamma^ R^2 (raw range)                      */
  KDA_WEIGHT_REL_RANGE = 3,     /* R~^2 (relative range)                       */
  KDA_WEIGHT_PERSISTENCE = 4,   /* w1 R~^2, w1 = 1/(1 - exp(-2 s^)) (DAMP's
                                   uncapped persistence, Related work)        */
  KDA_WEIGHT_WRITEBACK = 5,     /* h R~^2, h = 1/(1 - exp(-2 C s^)) with C the
                                   write-back interval (1 for kda_step)        */
  KDA_WEIGHT_NO_ERASE_RATE = 6, /* Gamma^ with r = 0, times R~^2              */
  KDA_WEIGHT_UNIFORM = 7,       /* equal keys: uniform widths (the remainder
                                   of the budget to the lowest rows)          */
  KDA_WEIGHT_DECAY = 8          /* Gamma^ alone, ranges ignored (decay-only
                                   allocation, Sec. 5, Effect of range
                                   normalization)                             */
} kda_weight_mode;

typedef struct {
  int32_t B;              /* sequences                                        */
  int32_t H;              /* heads per layer                                  */
  int32_t d_k;            /* rows (key channels): 64, 128 or 256 (256 needs
                             b_max <= 8)                                      */
  int32_t d_v;            /* columns (value channels): equal to d_k           */
  int32_t group_rows;     /* G: rows per output-normalisation group (Sec. 2,
                             Range normalization): divides d_k, or (groups
                             spanning heads, as Mamba-2's 12-head groups) a
                             multiple of d_k dividing H*d_k with
                             KDA_SCOPE_SEQUENCE                               */
  int32_t scope;          /* allocation scope: KDA_SCOPE_SEQUENCE = all H*d_k
                             rows of a sequence share the budget (the paper's
                             layer budget, Sec. 3); KDA_SCOPE_HEAD = per head */
  double mean_bits;       /* mean payload bits per element, in [b_min, b_max] */
  int32_t b_min, b_max;   /* width clamp, 1 <= b_min <= b_max <= 16 (Sec. 3)  */
  int32_t ema_span;       /* EMA span in tokens (Sec. 3: 64); 1 = one-token   */
  int32_t decay_per_head; /* 0: s is per row [.., H, d_k]; 1: one rate per
                             head [.., H] (Gated DeltaNet style, Sec. 1)      */
  int32_t state32;        /* 1: unquantised float32 state ("32-bit mode")     */
  int32_t no_erase;       /* 1: no erasure, a_t = 0 in eq. rule (Mamba-2):
                             S = D S + beta k v^T and no erase term in the
                             rate statistics and weights; 0: KDA/GDN erase */
  int32_t chunked;        /* kda_prefill only.  0: token-sequential float32
                             recurrence (bit-reproducible contract); 1: each
                             write-back interval in the chunked (WY/UT) form
                             of eq. rule on bf16 MFMA with float32
                             accumulation, every operand that is not exact
                             in bf16 split into hi and lo bf16 parts (three
                             products), so state and outputs agree with the
                             recurrence to float32-level accuracy (not bit
                             for bit), with C <= 64 and d_k <= 128.  The
                             write-back quantiser is the same in both modes. */
  int32_t head_units;     /* 1: allocation units are heads (Sec. 3, Allocation
                             units, Gated DeltaNet): one width per head from
                             the layer budget over the H heads of a sequence
                             (key: mean Gamma of the head's rows; R~ = 1),
                             FP16 scales per block of 32 rows of a column;
                             needs group_rows = d_k, KDA_SCOPE_SEQUENCE and
                             2 <= b_min <= b_max <= 8.  kda_step and
                             kda_prefill only (the two-phase step, pack,
                             unpack and kda_alloc_bits return
                             KDA_ERR_UNSUPPORTED).  Record layout: u32
                             tokens; u32 width (0 = zero state); 8 reserved
                             bytes; rate code u16 [d_k]; erase rate FP16
                             [d_k]; block scales FP16 [d_k/32][d_v]; at the
                             next multiple of 256 the code words as below
                             with every row of width b (row i at bit i b). */
  int32_t weight_mode;    /* allocation key (Sec. 5, Table ablate), a
                             kda_weight_mode; KDA_WEIGHT_EMA (0) is the
                             paper's method.  With head_units only the modes
                             that need no ranges (EMA, PERSISTENCE,
                             WRITEBACK, NO_ERASE_RATE, UNIFORM).            */
} kda_config;

/* Bytes of one (sequence, head) record slot; 0 if the config is invalid.
 * Quantised layout (little endian):
 *   u32 tokens seen; u32 reserved[3];
 *   widths: d_k 4-bit fields (b - 1), row i in byte i/2, low nibble if i even;
 *   scale FP16 [d_k]; rate code u16 [d_k]; erase rate FP16 [d_k];
 *   at the next multiple of 256: code words u32 [ceil(d_k*b_max/32)][d_v];
 *   column j is a bit stream of the rows' b_i-bit two's complement codes in
 *   row order, least significant bit first, so row i starts at bit
 *   sum_{i'<i} b_i' (prefix sums of widths, Sec. 3); bit p of column j is bit
 *   p%32 of word [p/32][j].  One-bit rows store 1 for a negative value and
 *   scale = mean |x|.
 * 32-bit mode: the float32 state, row-major [d_k][d_v]. */
size_t kda_record_bytes(const kda_config* cfg);

/* Bytes of workspace kda_step / kda_prefill / kda_alloc_bits need.  Any
 * contents are valid on entry. */
size_t kda_workspace_bytes(const kda_config* cfg);

/* Static description of a status code. */
const char* kda_status_str(int status);

/* Windowed observability-Gramian row weights (Prop. 1, eq. gram, with the
 * diagonal erase approximation of Sec. 2, Approximate erasure rate):
 *   lambda_t,i = exp(-2 s_t,i - beta_t (2 - beta_t) k_t,i^2)   (no erase
 *                term with no_erase),
 *   A_0 = 0, A_t = lambda_t (chi_{t-1} + A_{t-1}),
 *   gamma_i = (1/W) sum_{t=1}^{W-1} q_t,i^2 A_t,i,
 * chi_tau = 1 when a write-back follows token tau ((tau+1) % C == 0).
 * In:  q, k [B][W][H][d_k] f32; s [B][W][H][d_k] f32 (or [B][W][H] with
 *      decay_per_head); beta [B][W][H] f32.  W >= 1, C >= 1.
 * Out: gamma [B][H][d_k] f64. */
int kda_weights(const kda_config* cfg, int32_t W, int32_t C, const float* q,
                const float* s, const float* beta, const float* k,
                double* gamma, void* stream);

/* Exact Gramian row weights (Prop. 1, eq. gram) over a window, with the full
 * transition F_t = (I - beta_t k_t k_t^T) diag(exp(-s_t)) instead of the
 * diagonal erase approximation: backward over the window,
 *   M <- F_t^T (q_t q_t^T + M) F_t   for t = W-1 down to 1,
 *   gamma_i = (1/W) sum_t chi_{t-1} M_ii,
 * chi as in kda_weights (the exact-Gramian allocation the paper compares its
 * estimate against, Sec. 3, State bit allocation).  Float64, O(d_k^2) per
 * token and head.  Arguments and layouts as kda_weights; d_k <= 128
 * (KDA_ERR_UNSUPPORTED otherwise: the matrix is held in registers). */
int kda_weights_exact(const kda_config* cfg, int32_t W, int32_t C, const float* q,
                      const float* s, const float* beta, const float* k,
                      double* gamma, void* stream);

/* Bit allocation (Sec. 3, eq. weight and eq. alloc, rounded, clipped and
 * adjusted to the budget): R~ = R / RMS_group(R), c = gamma * R~^2, widths
 * minimising sum c_i 2^(-2 b_i) with sum b_i = floor(mean_bits*N + 0.5) over
 * each scope unit of N rows; ties to the lower row index.
 * Groups of G rows may span heads (see group_rows).
 * In:  gamma [B][H][d_k] f64 (>= 0); R [B][H][d_k] f32 row absolute maxima.
 * Out: bits [B][H][d_k] u8.  ws: a workspace of kda_workspace_bytes (the
 * weights are formed in LDS; it is checked, not written). */
int kda_alloc_bits(const kda_config* cfg, const double* gamma, const float* R,
                   uint8_t* bits, void* ws, void* stream);

/* Quantise and pack states (Sec. 3, Levels and storage).
 * In:  S [B][H][d_k][d_v] f32; bits [B][H][d_k] u8 in [b_min, b_max];
 *      s_hat [B][H][d_k] f64 decay rates (stored as 16-bit log-uniform codes,
 *      Sec. 3, Decay-gate quantization); r [B][H][d_k] f64 erase rates
 *      (stored as FP16); tokens_seen is written to every slot header.
 * Out: records, B*H slots.  Not available in 32-bit mode. */
int kda_pack_state(const kda_config* cfg, const float* S, const uint8_t* bits,
                   const double* s_hat, const double* r, uint32_t tokens_seen,
                   void* records, void* stream);

/* Decode records (Sec. 3, Levels and storage: x^ = code * Delta per row,
 * one-bit rows +-mean|x|; rows addressed by prefix sums of the widths; rates
 * from their log-uniform codes, Sec. 3, Decay-gate quantization).
 * Out (each may be NULL): S [B][H][d_k][d_v] f32
 * dequantised state; bits [B][H][d_k] u8; s_hat [B][H][d_k] f64 decoded
 * rates; r [B][H][d_k] f64 decoded erase rates.  In 32-bit mode only S.
 * Records are only read; a zero slot decodes to the zero state. */
int kda_unpack_state(const kda_config* cfg, const void* records, float* S,
                     uint8_t* bits, double* s_hat, double* r, void* stream);

/* One decode token for B x H heads with a write-back (C = 1): the gated
 * delta rule of Sec. 2, eq. rule (KDA erase and write vectors, or none with
 * no_erase), the output o = S^T q read before quantisation (Sec. 2,
 * Accumulated readout error), then the write-back of Sec. 3: EMA rate
 * statistics and weights (eq. weight), range normalisation, widths in the
 * layer budget (eq. alloc), the fitted row quantiser (Levels and storage)
 * and the record rewritten in place.
 * In:  q, k [B][H][d_k] f32 (k unit norm); v [B][H][d_v] f32;
 *      s [B][H][d_k] f32 (or [B][H] with decay_per_head), s > 0;
 *      beta [B][H] f32; gamma: NULL to weight rows by the EMA estimate of
 *      eq. weight, else [B][H][d_k] f64 weights (e.g. from kda_weights).
 * In/out: records.  Out: o [B][H][d_v] f32, read before quantisation. */
int kda_step(const kda_config* cfg, void* records, const float* q,
             const float* k, const float* v, const float* s, const float* beta,
             const double* gamma, float* o, void* ws, void* stream);

/* kda_step without a workspace argument and without any device allocation,
 * for callers that cannot allocate: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.  The scratch kda_step takes
 * from `ws` comes from a file-scope device array of the library instead (one
 * per GPU, 16 MiB, kda_step_noalloc_max_bytes(), held until the process
 * ends; its address is looked up once per device).  Same arguments, results
 * and errors as kda_step, except: d_k <= 128 with per-row units (head_units
 * or d_k = 256 give KDA_ERR_UNSUPPORTED; 32-bit mode needs no scratch and is
 * forwarded to kda_step), and a configuration whose scratch exceeds 16 MiB
 * (the decode layer B=64, H=32, d_k=128 needs about 10.3 MiB) gives
 * KDA_ERR_WORKSPACE before anything is launched.  Every call on one GPU
 * shares that GPU's array, which keeps the previous call's contents (any
 * contents are valid on entry): calls that overlap on one GPU (concurrent
 * streams, or host threads without ordering) race and must not be made. */
int kda_step_noalloc(const kda_config* cfg, void* records, const float* q,
                     const float* k, const float* v, const float* s,
                     const float* beta, const double* gamma, float* o,
                     void* stream);
size_t kda_step_noalloc_max_bytes(void);

/* kda_step in two phases, for callers that overlap a layer's write-back with
 * later work (the outputs precede the quantisation, Sec. 2, Accumulated
 * readout error, so the next layer needs only the first phase).  The first
 * phase is Sec. 2, eq. rule and the rate statistics, weights and widths of
 * Sec. 3 (eq. weight, eq. alloc); the second is Sec. 3, Levels and storage.
 * kda_step_outputs: the token's recurrence, outputs o, rate statistics,
 *   weights and widths; what the write-back needs of the state after the
 *   token is left in ws (the token's vectors for d_k <= 128, else the float32
 *   state).  Records are only read.  Arguments as kda_step.
 * kda_step_writeback: quantise the state after the token (rebuilt from the
 *   unchanged records and ws) with those widths and rewrite the records in
 *   place.  Must follow kda_step_outputs of the same records and ws (stream
 *   order or an event), before ws or the records are used by another call.  Not available in 32-bit mode (kda_step_outputs
 *   then does the whole step and kda_step_writeback returns KDA_OK).
 * kda_step(...) is kda_step_outputs(...) then kda_step_writeback(...) on one
 * stream. */
int kda_step_outputs(const kda_config* cfg, void* records, const float* q,
                     const float* k, const float* v, const float* s,
                     const float* beta, const double* gamma, float* o, void* ws,
                     void* stream);
int kda_step_writeback(const kda_config* cfg, void* records, void* ws, void* stream);

/* Per-token decay-gate quantisation (Sec. 3, Decay-gate quantization): for
 * every (sequence, token, head), the d_k rates are coded with 2^bits levels
 * uniform in log s (KDA_GATES_LOG) or in g = -s (KDA_GATES_LINEAR, the
 * comparison of that passage) over the range of the head's channels at that
 * token, and replaced by their dequantised values (float64 arithmetic:
 * x = log s or s, step = (max x - min x) / (2^bits - 1), code =
 * clamp(rne((x - min x) / step), 0, 2^bits - 1), x^ = min x + code step).
 * In: s [B][T][H][d_k] f32 (per-row decay; decay_per_head is unsupported),
 * 1 <= bits <= 16.  Out: s_out, same layout (may equal s).  The quantised
 * gates feed kda_prefill / kda_step like any rates. */
enum { KDA_GATES_LOG = 0, KDA_GATES_LINEAR = 1 };
int kda_gate_quant(const kda_config* cfg, int32_t T, int32_t bits, int32_t mode, const float* s,
                   float* s_out, void* stream);

/* Prefill of T tokens with a write-back after every C-th token and after the
 * last one (Sec. 2: the state is written back once per prefill chunk; the
 * recurrence is eq. rule and each write-back the quantiser of Sec. 3, as in
 * kda_step).  With cfg->chunked, each write-back interval is evaluated in the
 * chunked (WY/UT) form of eq. rule; C must then be at most 64 (KDA_ERR_ARG
 * otherwise) and the workspace (kda_workspace_bytes of the same config) also
 * holds the per-chunk records of two groups of up to 16 chunks per head
 * (153 600 bytes per chunk and head at d_k = 128).  All work is enqueued on
 * `stream`.
 * In:  q, k [B][T][H][d_k] bf16 (raw 16-bit patterns); v [B][T][H][d_v] bf16;
 *      s [B][T][H][d_k] f32 (or [B][T][H]); beta [B][T][H] f32; gamma as in
 *      kda_step.  In/out: records.  Out: o [B][T][H][d_v] f32. */
int kda_prefill(const kda_config* cfg, int32_t T, int32_t C, void* records,
                const uint16_t* q, const uint16_t* k, const uint16_t* v,
                const float* s, const float* beta, const double* gamma,
                float* o, void* ws, void* stream);

/* kda_prefill with a second stream of the caller's (Sec. 2, chunked
 * prefill as above).  With cfg->chunked and more than one chunk, the
 * chunk preparation of later groups of chunks runs on aux_stream beside the
 * current group's write-back intervals on `stream`: the call orders the two
 * streams with events it creates and destroys itself, and before returning
 * (on every path, errors included) makes `stream` wait for all of its work on
 * aux_stream, so the call's work is complete in `stream` order and, under
 * graph capture on `stream`, every branch on aux_stream is joined back.  The
 * caller owns aux_stream and must not enqueue other work on it during the
 * call.  aux_stream NULL or equal to `stream`: the single-stream schedule of
 * kda_prefill.  Without cfg->chunked aux_stream is not used.  The library
 * keeps no streams, events or locks between calls. */
int kda_prefill_aux(const kda_config* cfg, int32_t T, int32_t C, void* records,
                    const uint16_t* q, const uint16_t* k, const uint16_t* v,
                    const float* s, const float* beta, const double* gamma,
                    float* o, void* ws, void* stream, void* aux_stream);

/* Diagnostics: per-kernel timing and work counts.  With KDA_PROFILE_EVENTS,
 * every kernel a call enqueues is bracketed by two hipEvents recorded on the
 * call's stream (host-side runtime objects from a reusable pool).  With
 * KDA_PROFILE_COUNTERS, the quantiser counts its clip-factor evaluations into
 * an 8-byte device counter that the first such call allocates (the only
 * device allocation the library makes; it lives until the process ends; the
 * counting itself slows the quantiser down).  flags = 0 turns both off.  Not
 * thread safe; meant for single-threaded benchmark drivers. */
enum { KDA_PROFILE_EVENTS = 1, KDA_PROFILE_COUNTERS = 2 };
int kda_profile_enable(int flags);

/* Synchronise the device, then report and clear the number of (row segment of
 * 64 columns) x (clip-factor candidate) evaluations counted while profiling
 * was enabled.  Host pointer. */
int kda_profile_counters(unsigned long long* fit_evals);

/* Wait for the last recorded event, then report per kernel kind (static
 * strings such as "stats", "alloc", "requant") the summed milliseconds and
 * launch counts since the previous read, and forget them.  Host pointers;
 * kinds/ms/counts hold up to max_kinds entries (each may be NULL);
 * *n_kinds receives the number of kinds seen. */
int kda_profile_read(int max_kinds, const char** kinds, double* ms, int* counts,
                     int* n_kinds);

#ifdef __cplusplus
}
#endif
#endif /* KDA_H_ */
