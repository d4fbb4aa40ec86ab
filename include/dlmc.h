/*
 * dlmc.h -- lossless compression with a masked diffusion language model on
 * AMD MI355X (gfx950).  C ABI of libdlmc.so.
 *
 * Method: "Diffuse to Compress: Leveraging Diffusion LMs for Lossless
 * Compression" (Nardone, Ferragina).  A sequence is split into independent
 * non-overlapping windows ("chunks", Implementation Details).  Each chunk
 * starts fully masked and is reconstructed over several inference steps
 * (Diffusion-Based Compression Pipeline): one forward pass of a masked
 * diffusion LM (Definition 3) gives a distribution at every masked position,
 * the entropy-based commitment schedule (Symbol Commitment Schedules, item 3)
 * picks positions, their symbols are coded with their predicted distributions
 * by a statistical coder, and the symbols are revealed.  The schedule is
 * deterministic, so the decoder replays it from the header alone (the remark
 * closing Symbol Commitment Schedules).
 *
 * Conventions for every call:
 *   - the return value is a dlmc_status: 0 on success, a negative code on
 *     error; no C++ exception crosses the ABI; dlmc_last_error() gives a
 *     thread-local message for the last failure on the calling thread;
 *   - "host" pointers are caller-owned CPU memory, read or written during the
 *     call only and never retained;
 *   - "device" pointers are caller-owned GPU memory on the model's device
 *     (e.g. torch tensors); the library reads / writes them on the model's
 *     stream and never frees them;
 *   - a dlmc_model handle is not thread safe: use one handle per host thread.
 */
#ifndef DLMC_H
#define DLMC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t dlmc_status;
#define DLMC_OK 0
#define DLMC_E_INVAL -1   /* bad argument or unsupported configuration */
#define DLMC_E_NOMEM -2   /* device or host allocation failed */
#define DLMC_E_DEVICE -3  /* HIP runtime error */
#define DLMC_E_FORMAT -4  /* not a dlmc container, or made by another model */
#define DLMC_E_CORRUPT -5 /* bitstream fails to decode, or CRC mismatch */
#define DLMC_E_BUFFER -6  /* output buffer too small; required size reported */
#define DLMC_E_NUMERIC -7 /* non-finite logits or entropies */

#define DLMC_FFN_GELU 0   /* x W1^T -> exact-erf GELU -> W2^T          */
#define DLMC_FFN_SWIGLU 1 /* (silu(x Wg^T) * x Wu^T) Wd^T               */
#define DLMC_NORM_LAYER 0 /* LayerNorm, gain 1, bias 0                  */
#define DLMC_NORM_RMS 1   /* RMSNorm, gain 1                            */
#define DLMC_DTYPE_F32 0  /* fp32 weights, activations and accumulation */
#define DLMC_DTYPE_BF16 1 /* bf16 weights and GEMM inputs, fp32 accumulate,
                             fp32 residual stream, norms, softmax, logits */

/* Shape of the masked diffusion LM (Definition 3).  vocab = |Sigma|; the
 * input-only [MASK] token id is vocab.  Weights are random: tensor entries
 * are uniform on [-2^-e, 2^-e) from a counter-based generator (see
 * dlmc_model_create) with e = the matching *_exp field. */
typedef struct dlmc_model_config {
  uint32_t struct_size; /* sizeof(dlmc_model_config) */
  int32_t n_layers;     /* >= 0 */
  int32_t d_model;      /* multiple of 128 (bf16) or 16 (f32) */
  int32_t n_heads;      /* d_model / n_heads in {64, 128} (bf16), <= 128 (f32) */
  int32_t d_ffn;        /* multiple of 64 (bf16) or 16 (f32) */
  int32_t vocab;        /* |Sigma| >= 2; 2^cdf_bits must exceed it */
  int32_t ffn_kind;     /* DLMC_FFN_* */
  int32_t norm_kind;    /* DLMC_NORM_* */
  int32_t dtype;        /* DLMC_DTYPE_* */
  float rope_theta;     /* rotary base (rotate-half pairing of i, i + d_head/2) */
  float norm_eps;
  int32_t embed_exp, attn_exp, ffn_in_exp, ffn_out_exp, head_exp;
  int32_t max_chunk; /* largest chunk length any call will use */
  int32_t max_batch; /* largest number of chunks per forward pass */
} dlmc_model_config;

/* Commitment schedule and coder parameters (stored in the container header).
 * Entropy-based schedule: commit every masked position whose entropy (bits)
 * is <= tau_bits; if fewer than m_min qualify commit the m_min lowest; never
 * more than m_max; ties by lower position; all remaining positions if fewer
 * than m_min are masked.  tau_bits = -INFINITY with m_min = m_max = k is the
 * fixed-k rule.  Committed symbols are coded in ascending position order. */
typedef struct dlmc_codec_params {
  uint32_t struct_size; /* sizeof(dlmc_codec_params) */
  int32_t chunk_len;    /* window length w, 1..max_chunk */
  /* entropy schedule (Symbol Commitment Schedules, item 3): commit every
   * masked position with entropy <= tau_bits, at least m_min (the lowest),
   * at most m_max; tau_bits = -inf with m_min = m_max = k is fixed-k.  For the
   * block schedules m_max is the per-pass capacity (no block may exceed it). */
  float tau_bits;
  int32_t m_min; /* >= 1 */
  int32_t m_max; /* m_min..1024 */
  int32_t cdf_bits;   /* P: CDF precision, 2^P > vocab; range coder: P <= coder_bits - 16,
                         rANS: P <= 31 */
  int32_t coder_bits; /* W: range coder width, 32 or 64 (rANS: ignored, 64) */
  int32_t batch;      /* chunks per forward, 1..max_batch; does not change the output */
  int32_t flags;      /* DLMC_FLAG_* */
  int32_t schedule;   /* DLMC_SCHED_* */
  int32_t blocks;     /* uniform block schedule: K >= 1 blocks per chunk
                         (item 1: u = floor(n/K) left to right, the remainder
                         n mod K on the last block, K > n read as K = n) */
  int32_t u1;         /* progressive schedule (item 2): first block >= 1 */
  double growth;      /* progressive: ratio r > 0; u_k = round-half-up(u1 r^(k-1)),
                         r^(k-1) by repeated fp64 multiplication, >= 1 per pass,
                         the last block cut to what remains */
  int32_t coder;      /* DLMC_CODER_* */
  int32_t context;    /* initial context (Initial Context Strategies): c >= 0
                         symbols per chunk left visible and stored in the chunk
                         payload (min(c, chunk length) for a short chunk) */
  int32_t context_kind; /* DLMC_CONTEXT_* */
  int32_t rank_compressor; /* DLMC_CODER_RANK: DLMC_RANKC_* applied to the
                              container's payload section as one block */
  uint64_t context_seed; /* random context of chunk i: the c positions with the
                            smallest keys splitmix64(splitmix64(seed + i) + p) */
  int32_t rank_level;    /* compressor level: zlib 0..9, lzma preset 0..9,
                            zstd 1..22, none 0 */
  int32_t reserved;      /* 0 */
} dlmc_codec_params;

#define DLMC_SCHED_ENTROPY 0
#define DLMC_SCHED_UNIFORM 1
#define DLMC_SCHED_PROGRESSIVE 2
#define DLMC_CODER_RANGE 0
#define DLMC_CODER_RANS 1
/* symbol ranking (Definition of Symbol Ranking): the rank of every coded
 * symbol in the list ordered by non-increasing probability (equal
 * probabilities by token id), written as unsigned LEB128 varints */
#define DLMC_CODER_RANK 2
#define DLMC_RANKC_NONE 0
#define DLMC_RANKC_ZLIB 1
#define DLMC_RANKC_LZMA 2 /* xz container, CRC-64 check */
#define DLMC_RANKC_ZSTD 3
#define DLMC_CONTEXT_CONTIGUOUS 0 /* the first c positions */
#define DLMC_CONTEXT_RANDOM 1     /* c seeded-random positions */
/* the c positions with the highest Attention Rollout flow into the masked
 * positions of two extra passes (even, then odd positions masked); each
 * position is scored in the pass where it is visible, ties by position */
#define DLMC_CONTEXT_ATTENTION 2

#define DLMC_FLAG_CRC 1 /* store and check a CRC-32 of every chunk's tokens */

typedef struct dlmc_model dlmc_model;
typedef struct dlmc_session dlmc_session;

/* ---- model ------------------------------------------------------------ */

/* Create a model on HIP device `device` and generate its weights from
 * `seed`: tensor t (embedding 1, head 2, layer l kind k -> 16 + 16 l + k with
 * q,k,v,o,ffn_in,ffn_up,ffn_out = 0..6; all [out, in] row-major, embedding
 * [vocab+1, d]) has entries w_i = ((u_i >> 40) - 2^23) 2^(-23-e) with
 * u_i = splitmix64(splitmix64(seed ^ t*0x9E3779B97F4A7C15) + i), rounded to
 * nearest-even bf16 for bf16 models.  The library owns the weights and the
 * workspace for max_batch chunks of max_chunk tokens.
 * Errors: E_INVAL (config), E_NOMEM, E_DEVICE. */
dlmc_status dlmc_model_create(const dlmc_model_config* cfg, uint64_t seed, int32_t device,
                              dlmc_model** out);
/* Free the model and all its device memory.  NULL is ignored. */
void dlmc_model_destroy(dlmc_model* model);
/* Use `hip_stream` (a hipStream_t, e.g. torch.cuda.current_stream().cuda_stream)
 * for all device work of this model; NULL selects the library's own stream. */
dlmc_status dlmc_set_stream(dlmc_model* model, void* hip_stream);

/* ---- compression ------------------------------------------------------- */

/* Container (version 3, little endian).  The header stores the window
 * length and every schedule parameter, so that the decoder replays the
 * encoder's decisions from it alone (Implementation Details; the remark
 * closing Symbol Commitment Schedules):
 *   0 magic "DLMC", 4 version, 8 header bytes, 12 flags, 16 model hash
 *   (FNV-1a 64 of the config fields that change results and the seed),
 *   24 seed, 32 n_tokens, 40 n_chunks, 48 chunk_len, 52 cdf_bits,
 *   56 coder_bits, 60 m_min, 64 m_max, 68 tau_bits (f32), 72 batch,
 *   76 schedule, 80 blocks, 84 u1, 88 growth (f64), 96 coder, 100 context,
 *   104 context_kind, 108 rank_compressor, 112 rank_level, 116 reserved,
 *   120 numerics id (dlmc_numerics_id), 128 first chunk held, 136 number of
 *   chunks held (count); then u64 offsets[count + 1] of the held chunks'
 *   payloads in the payload section, then (DLMC_FLAG_CRC) u32 CRC-32 of each
 *   held chunk's tokens (as int32), then the payload section.  A chunk's
 *   payload is its initial context (c u16 positions ascending, then c u32
 *   symbols) followed by its coder's bytes; the symbol ranking back end
 *   stores the whole payload section compressed as one block. */

/* Worst-case container size in bytes for n_tokens tokens. */
dlmc_status dlmc_encode_bound(const dlmc_model* model, const dlmc_codec_params* codec,
                              uint64_t n_tokens, uint64_t* bytes);
/* Compress host tokens[0..n) (each in [0, vocab)) into the host buffer
 * out[0..cap).  On E_BUFFER *out_len holds the required size. */
dlmc_status dlmc_encode(dlmc_model* model, const dlmc_codec_params* codec,
                        const int32_t* tokens, uint64_t n, uint8_t* out, uint64_t cap,
                        uint64_t* out_len);
/* Encode only the chunks [first_chunk, first_chunk + n_chunks) of host
 * tokens[0..n) (chunk i covers tokens [i w, min(n, (i + 1) w)), w =
 * codec->chunk_len) into a partial container that holds them under their
 * global indices.  Windows are independent (Implementation Details: non-
 * overlapping windows can be processed in parallel, e.g. one range per GPU),
 * so the chunk payloads are byte-identical to those of dlmc_encode of the
 * whole input.  n_chunks = UINT64_MAX means "to the last chunk"; a range
 * outside the input's chunks is E_INVAL.  Partial containers are combined
 * with dlmc_merge; dlmc_decode accepts only complete containers.  The bound
 * call gives the worst-case size of such a partial container. */
dlmc_status dlmc_encode_range(dlmc_model* model, const dlmc_codec_params* codec,
                              const int32_t* tokens, uint64_t n, uint64_t first_chunk,
                              uint64_t n_chunks, uint8_t* out, uint64_t cap, uint64_t* out_len);
dlmc_status dlmc_encode_range_bound(const dlmc_model* model, const dlmc_codec_params* codec,
                                    uint64_t n_tokens, uint64_t first_chunk, uint64_t n_chunks,
                                    uint64_t* bytes);
/* Combine n_parts host containers (parts[i] of lens[i] bytes, in any order)
 * of the same input, model, build and codec parameters whose chunk ranges
 * tile all of the input's chunks into one complete container in out[0..cap),
 * byte-identical to dlmc_encode of the whole input.  No GPU is used.
 * E_FORMAT if the parts disagree in any header field, overlap, or leave a
 * chunk out; E_BUFFER as for dlmc_encode. */
dlmc_status dlmc_merge(const uint8_t* const* parts, const uint64_t* lens, int32_t n_parts,
                       uint8_t* out, uint64_t cap, uint64_t* out_len);
/* Number of tokens a container holds (reads the header only; E_FORMAT, also
 * for a container made by a build with another numerics identity). */
dlmc_status dlmc_decode_size(const uint8_t* in, uint64_t len, uint64_t* n_tokens);
/* The 64-bit numerics identity of this build: a hash of the library's source
 * code and compile flags.  Every container records the identity of the build
 * that made it, and a build with another identity refuses to decode it
 * (E_FORMAT): the decoder must replay the encoder's decisions exactly (the
 * remark closing Symbol Commitment Schedules), and kernels that round
 * differently could take other decisions. */
dlmc_status dlmc_numerics_id(uint64_t* id);
/* Decompress host container in[0..len) into host tokens[0..cap).  The codec
 * parameters come from the header; the batch used is `batch` when > 0, else
 * the header's.  The payload section is copied to device memory once and,
 * with the range coder or rANS, every pass's symbols are decoded on the
 * device (one wave per chunk of the batch, the host decoders' integer
 * arithmetic), so CDF rows never leave the GPU.  E_FORMAT if the container
 * was made by a model with another configuration or seed, or its header is
 * inconsistent with its length; E_CORRUPT on an undecodable stream or CRC
 * mismatch; E_BUFFER if cap is too small (*n = required, checked before any
 * allocation). */
dlmc_status dlmc_decode(dlmc_model* model, const uint8_t* in, uint64_t len, int32_t batch,
                        int32_t* tokens, uint64_t cap, uint64_t* n);

/* Streaming form of dlmc_encode: one call of dlmc_encoder_step runs exactly
 * one masked-diffusion pass over the current batch of chunks (forward,
 * entropy, selection, CDFs, coding, reveal).  `tokens` is copied at begin. */
dlmc_status dlmc_encoder_begin(dlmc_model* model, const dlmc_codec_params* codec,
                               const int32_t* tokens, uint64_t n, dlmc_session** out);
/* *done = 1 once every chunk is coded; *coded (optional) += symbols coded. */
dlmc_status dlmc_encoder_step(dlmc_session* s, int32_t* done, uint64_t* coded);
/* Finish (running any remaining passes) and write the container. */
dlmc_status dlmc_encoder_finish(dlmc_session* s, uint8_t* out, uint64_t cap, uint64_t* out_len);
void dlmc_session_destroy(dlmc_session* s);

/* Per (chunk, pass) trace of encode and decode (arrays valid during the
 * call only): the n_sel committed positions pos[] (ascending), their
 * entropies in bits, the coded pairs coded[2 j], coded[2 j + 1] of position
 * pos[j] -- the interval (start, freq) of its symbol in the 2^cdf_bits total
 * for the range and rANS coders, (rank, symbol) for symbol ranking -- and an
 * FNV-1a 64 hash of the committed rows' integer CDFs (of the coded symbols
 * for symbol ranking).  dir = 0 encode, 1 decode.  Encode and decode of the
 * same container report identical traces.  NULL disables. */
typedef void (*dlmc_trace_fn)(void* user, int32_t dir, uint64_t chunk, int32_t pass,
                              int32_t n_sel, const int32_t* pos, const float* entropy_bits,
                              const uint32_t* coded, uint64_t cdf_hash);
dlmc_status dlmc_set_trace(dlmc_model* model, dlmc_trace_fn fn, void* user);

/* ---- stage hooks (device pointers; tests and benchmarks) ---------------- */

/* Test hook for the error path of non-finite model output: while `on` is
 * nonzero, every forward pass of the model writes a NaN into the final-norm
 * input of its first LM-head row, so that row's logits and entropy are
 * non-finite and encoding fails with E_NUMERIC. */
dlmc_status dlmc_test_inject_nonfinite(dlmc_model* model, int32_t on);

/* Test hook for the deferred LM-head logits of the entropy schedule (bf16
 * models).  With many masked rows, the head writes only each row's entropy
 * statistics (Schedules, item 3) and the logits of the rows committed in the
 * pass are computed after the selection, which gives the same bits as storing
 * them all.  mode 0 (default): decided per pass by estimated cost; 1: always
 * deferred; 2: never.  Payloads do not depend on the mode.  E_INVAL for
 * another mode. */
dlmc_status dlmc_test_head_logits(dlmc_model* model, int32_t mode);

/* Test hook (host only, no GPU needed): the tile shape the bf16 GEMM chooses
 * for an M x N x K product with epilogue `epi` (0 fp32 store, 1 residual
 * update, 2 QKV with rotary, 3 GELU, 4 SwiGLU; d_model is the QKV
 * epilogue's model width, else unused).  *kind: 0 128 x 128 tiles, 1
 * 192 x 128 tiles (two blocks per CU), 2 the 4-wave kernel with columns
 * [0, *split) on 256 x 256 tiles and [*split, N) on 256 x 128 tiles.  The
 * choice never changes a result; the GEMMs run in the forward pass of
 * Definition 3.  E_INVAL for sizes the GEMM does not take (K % 64 != 0,
 * M, N < 1, paired epilogues with N % 128 != 0) or a NULL output. */
dlmc_status dlmc_test_gemm_tiles(int32_t M, int32_t N, int32_t K, int32_t epi, int32_t d_model,
                                 int32_t* kind, int32_t* split);

/* One forward pass (Definition 3) over device state[B*T] (int32, MASK =
 * vocab).  Writes the fp32 logits at the masked positions, in ascending
 * (chunk, position) order, to logits[n_rows * vocab], their flat indices
 * b*T + t to rows[n_rows], and n_rows to n_rows[0] (all device).  logits
 * must hold B*T*vocab floats, rows B*T ints. */
dlmc_status dlmc_forward_logits(dlmc_model* model, const int32_t* state, int32_t B, int32_t T,
                                float* logits, int32_t* rows, int32_t* n_rows);
/* Entropy (bits) and max of every row of device logits[n_rows * vocab], and
 * the integer CDF of every row at precision cdf_bits: g[n_rows*vocab] =
 * floor(exp(l - max) 2^24) and cdf[n_rows*(vocab+1)]; g and cdf may be NULL. */
dlmc_status dlmc_entropy_cdf(dlmc_model* model, const float* logits, int32_t n_rows,
                             int32_t cdf_bits, float* entropy_bits, float* row_max,
                             uint32_t* g, uint32_t* cdf);
/* dlmc_entropy_cdf for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments and results, bit for bit; no hipMalloc,
 * hipFree or other allocating call: the CDF's per-row tables and segment
 * partials live in the library's static device scratch of DLMC_SCRATCH_BYTES
 * per GPU (held by each GPU the library runs on until the process ends),
 * which must hold 8 n_rows bytes rounded up to 256 plus
 * 20 n_rows ceil(vocab / 4096) bytes when a CDF is asked for (about 6600
 * rows at vocab 126464); larger requests fail with E_INVAL before any work.
 * Like dlmc_entropy_cdf it returns once its work on the model's stream is
 * complete.  Every call on a GPU shares that GPU's scratch, so calls that
 * overlap in time on one GPU (other host threads, other model handles)
 * race: serialise them. */
#define DLMC_SCRATCH_BYTES (4u << 20)
dlmc_status dlmc_entropy_cdf_noalloc(dlmc_model* model, const float* logits, int32_t n_rows,
                                     int32_t cdf_bits, float* entropy_bits, float* row_max,
                                     uint32_t* g, uint32_t* cdf);
/* The commitment schedule on device entropies: rows[n_rows] are flat b*T+t
 * indices ascending (as from dlmc_forward_logits) with entropies H[n_rows].
 * Writes per chunk b the committed positions sel_pos[b*m_max + j], their
 * indices into rows sel_row[b*m_max + j] and the count n_sel[b]. */
dlmc_status dlmc_select(dlmc_model* model, const float* entropy_bits, const int32_t* rows,
                        int32_t n_rows, int32_t B, int32_t T, float tau_bits, int32_t m_min,
                        int32_t m_max, int32_t* sel_pos, int32_t* sel_row, int32_t* n_sel);
/* Symbol ranking on device logits[n_rows * vocab] (Definition of Symbol
 * Ranking; equal probabilities ordered by token id): rank[i] of sym[i] in row
 * i, and the inverse, sym[i] of rank[i] (0 <= rank < vocab; device int32
 * arrays of n_rows, n_rows <= 65535). */
dlmc_status dlmc_rank_rows(dlmc_model* model, const float* logits, int32_t n_rows,
                           const int32_t* sym, int32_t* rank);
dlmc_status dlmc_select_rank_rows(dlmc_model* model, const float* logits, int32_t n_rows,
                                  const int32_t* rank, int32_t* sym);
/* Attention-based context scores of one chunk of host tokens[0..T) into
 * host scores[0..T) (two extra forward passes, T <= max_chunk). */
dlmc_status dlmc_context_scores(dlmc_model* model, const int32_t* tokens, int32_t T, float* scores);
/* Copy weight tensor `tensor_id` (ids as in dlmc_model_create) to host dst in
 * its canonical [out, in] layout: bf16 bit patterns (uint16) or fp32. */
dlmc_status dlmc_weight_copy(dlmc_model* model, int32_t tensor_id, void* dst, uint64_t bytes);

/* Stage timing for benchmarks: every launch of a stage whose bit is set in
 * `stage_mask` (bit s = DLMC_STAGE_s; DLMC_PROFILE_ALL for all, 0 to stop) is
 * bracketed by HIP events on the model's stream, and the stage's algorithmic
 * work per launch (flops for GEMMs and attention, HBM bytes for the memory
 * bound stages) is accumulated.  Each call resets the counters.  Events cost
 * a little time per launch, so a throughput measurement should time only the
 * stages it reports.  dlmc_profile_read synchronises the stream and returns,
 * for `stage` (DLMC_STAGE_*), the summed event time in ms, the number of
 * launches and the summed work. */
#define DLMC_STAGE_EMBED 0
#define DLMC_STAGE_NORM 1
#define DLMC_STAGE_QKV 2      /* QKV GEMM with rotary epilogue          */
#define DLMC_STAGE_ATTN 3     /* non-causal flash attention             */
#define DLMC_STAGE_OPROJ 4    /* O projection + residual                */
#define DLMC_STAGE_FFN_IN 5   /* FFN in (GELU / SwiGLU gate+up)         */
#define DLMC_STAGE_FFN_OUT 6  /* FFN out + residual                     */
#define DLMC_STAGE_HEAD 7     /* LM head at masked rows                 */
#define DLMC_STAGE_ENTROPY 8
#define DLMC_STAGE_SELECT 9
#define DLMC_STAGE_CDF 10
#define DLMC_STAGE_REVEAL 11   /* encode: (start, freq) gather; decode: entropy decoder; reveal */
#define DLMC_STAGE_COMPACT 12
#define DLMC_N_STAGES 13
#define DLMC_PROFILE_ALL ((1u << DLMC_N_STAGES) - 1u)
/* Flag bit of `stage_mask`: the per-layer stages (NORM inside the layers,
 * QKV, ATTN, OPROJ, FFN_IN, FFN_OUT) are timed in one layer per forward pass
 * only, layer f % n_layers in the f-th forward since the enable call; stages
 * outside the layer loop are timed as usual.  Cuts the event overhead 1 /
 * n_layers-fold for a throughput run that still reports a live average
 * launch duration. */
#define DLMC_PROFILE_ONE_LAYER (1u << 31)
dlmc_status dlmc_profile_enable(dlmc_model* model, uint32_t stage_mask);
dlmc_status dlmc_profile_read(dlmc_model* model, int32_t stage, double* ms_total,
                              uint64_t* launches, double* work);

/* ---- host range coder hooks (no GPU needed) ----------------------------- */

/* Range-code n symbol intervals [start_i, start_i + freq_i) of a 2^P total
 * with the W-bit coder used inside the container; writes the flushed stream. */
dlmc_status dlmc_rc_encode(const uint32_t* start, const uint32_t* freq, uint64_t n,
                           int32_t cdf_bits, int32_t coder_bits, uint8_t* out, uint64_t cap,
                           uint64_t* out_len);
/* Decode n symbols, symbol i with host cdf[i*(V+1) .. i*(V+1)+V]. */
dlmc_status dlmc_rc_decode(const uint8_t* in, uint64_t len, const uint32_t* cdf, uint64_t n,
                           int32_t V, int32_t cdf_bits, int32_t coder_bits, int32_t* sym);
/* rANS (the stream of a DLMC_CODER_RANS chunk payload after its context):
 * code n intervals, 1 <= P <= 31; decoding checks that the stream ends in
 * the coder's initial state (E_CORRUPT otherwise). */
dlmc_status dlmc_rans_encode(const uint32_t* start, const uint32_t* freq, uint64_t n,
                             int32_t cdf_bits, uint8_t* out, uint64_t cap, uint64_t* out_len);
dlmc_status dlmc_rans_decode(const uint8_t* in, uint64_t len, const uint32_t* cdf, uint64_t n,
                             int32_t V, int32_t cdf_bits, int32_t* sym);

/* ---- errors -------------------------------------------------------------- */
const char* dlmc_status_string(dlmc_status s);
const char* dlmc_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* DLMC_H */
