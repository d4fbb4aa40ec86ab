// Internal runtime objects behind the C ABI: the model (weights + workspace)
// and encode / decode sessions (the per-chunk pass loop).
#pragma once

#include <memory>
#include <vector>

#include "kernels.h"
#include "range_coder.h"
#include "rans_coder.h"

struct dlmc_model {
  dlmc_model_config cfg{};
  uint64_t seed = 0;
  int device = 0;
  hipStream_t stream = nullptr;      // stream in use
  hipStream_t own_stream = nullptr;  // library-created stream
  size_t esz = 2;                    // bytes per weight / GEMM-input element
  bool bf16 = true;
  int dh = 0;
  std::vector<void*> allocs;

  // weights (device): embedding [V+1, d]; per layer fused QKV [3d, d] (rotary
  // pairs adjacent for bf16), O [d, d], FFN in [F or 2F, d] (gate/up pairs
  // interleaved for bf16 SwiGLU), FFN out [d, F]; head [V, d]
  void* embed = nullptr;
  void* head = nullptr;
  struct Layer {
    void *wqkv, *wo, *win, *wout;
  };
  std::vector<Layer> layers;
  float* rope_cos = nullptr;  // [max_chunk, dh/2]
  float* rope_sin = nullptr;

  // workspace for max_batch * max_chunk rows
  int max_rows = 0, Tp_max = 0;
  float* x = nullptr;  // fp32 residual stream [rows, d]
  void *h = nullptr, *q = nullptr, *k = nullptr, *vt = nullptr, *attn = nullptr, *ffn = nullptr;
  float* tmp = nullptr;  // fp32 model only: [rows, max(3d, 2F)]
  void* hm = nullptr;    // final-norm rows of masked positions [rows, d]
  float* logits = nullptr;  // [rows, V]
  void* stats = nullptr;    // bf16 head: softmax statistics per 128-column group [rows, G]
  float *H = nullptr, *mx = nullptr;
  int32_t *rows = nullptr, *n_rows = nullptr, *chunk_off = nullptr, *chunk_cnt = nullptr;
  int32_t *state = nullptr, *err = nullptr;

  // selection buffers, grown on demand: max_batch * sel_cap slots
  int sel_cap = 0;
  int32_t *sel_pos = nullptr, *sel_row = nullptr, *n_sel = nullptr, *dec = nullptr;
  uint32_t *cdf = nullptr, *sym = nullptr;
  void* cdf_ws = nullptr;  // segment partials of the CDF kernels
  int64_t* slot_base = nullptr;
  int32_t* slot_rows = nullptr;  // slot_rows[i] = i: logits stored in slot order
  float* slot_mx = nullptr;      // row max of selection slot i (deferred head)
  int32_t* tokens_dev = nullptr;
  size_t tokens_cap = 0;

  void* scratch = nullptr;  // this device's copy of the library's static scratch
  bool inject_nan = false;  // test hook: a NaN into the first logit of every forward
  // Deferred logits.  head_slots (set by the caller of forward, 0 = never):
  // the selection slots whose logits a deferred head would recompute;
  // head_mode: 0 chooses by cost, 1 always defers, 2 never (test hook).
  // head_deferred: the last forward wrote only the entropy statistics.
  int head_slots = 0, head_mode = 0;
  bool head_deferred = false;
  dlmc_trace_fn trace = nullptr;
  void* trace_user = nullptr;

  // stage profiling (events bracket each stage launch while enabled)
  struct ProfRec {
    int stage;
    hipEvent_t a, b;
    double work;
  };
  uint32_t prof = 0;            // bit s set: stage s is timed
  bool prof_one_layer = false;  // per-layer stages timed in one layer per forward
  uint64_t prof_fwd = 0;        // forwards since profiling was enabled
  bool prof_gated = false;      // inside a layer that is not timed
  std::vector<ProfRec> prof_recs;
  std::vector<hipEvent_t> prof_pool;
  double prof_ms[DLMC_N_STAGES] = {}, prof_work[DLMC_N_STAGES] = {};
  uint64_t prof_n[DLMC_N_STAGES] = {};
  hipEvent_t prof_event();
  void prof_collect();
  void prof_reset();

  ~dlmc_model();
  void* dalloc(size_t bytes, bool zero = false);
  void dfree(void* p);
  void ensure_sel(int m_max);
  void ensure_tokens(size_t n);
  uint64_t hash() const;
  // One forward pass over state[B*T] (device): logits at masked rows into
  // logits_out (or the internal buffer), row ids and count likewise.  With
  // rows_given the head rows are the ones already in rows / n_rows (the
  // committed rows of a block schedule) instead of the masked rows.
  void forward(const int32_t* state, int B, int T, float* logits_out, int32_t* rows_out,
               int32_t* n_rows_out, int64_t rows_hint = -1, bool rows_given = false,
               float* attn_maps = nullptr);
  // attention-based context: per layer head-averaged attention maps of one
  // chunk (B = 1) written to attn_maps [L, T, T] by forward (the head is then
  // skipped); context_scores runs the two half-masked passes and returns the
  // rollout score of every position (host tokens and scores)
  float *ctx_maps = nullptr, *ctx_S = nullptr, *ctx_v = nullptr;
  int32_t* ctx_state = nullptr;
  int ctx_T = 0;
  void context_scores(const int32_t* tokens, int T, std::vector<float>& score);
  // entropy (bits) and max of the first n_rows[0] (at most n_max) head rows of
  // the last forward into H / mx: merged from the head's group statistics
  // (bf16), or from the stored logits (fp32); both give the same bits
  void row_stats(int n_max);
  // after a deferred head: the logits of the committed rows (sel_row /
  // n_sel, B chunks of m_max slots) into logits, in slot order
  void selected_logits(int B, int m_max);
  // row index of selection slot i in logits: sel_row, or the slot itself
  // after a deferred head
  const int32_t* logit_rows() const { return head_deferred ? slot_rows : sel_row; }
  // the row maxima the CDF reads at logit_rows()
  const float* logit_max() const { return head_deferred ? slot_mx : mx; }
};

namespace dlmc {
// Brackets one stage launch with events when the model's profiling is on.
struct StageTimer {
  dlmc_model* m;
  int stage;
  double work;
  hipEvent_t a = nullptr;
  StageTimer(dlmc_model* m_, int stage_, double work_) : m(m_), stage(stage_), work(work_) {
    if ((m->prof & (1u << stage_)) && !m->prof_gated) {
      a = m->prof_event();
      DLMC_HIP(hipEventRecord(a, m->stream));
    }
  }
  ~StageTimer() {
    if (a) {
      hipEvent_t b = m->prof_event();
      if (hipEventRecord(b, m->stream) == hipSuccess) m->prof_recs.push_back({stage, a, b, work});
    }
  }
};
}  // namespace dlmc

namespace dlmc {

// block compression of the symbol-ranking payload section (DLMC_RANKC_*)
bool rank_compressor_ok(int kind, int level);
std::vector<uint8_t> compress_block(int kind, int level, const std::vector<uint8_t>& in);
std::vector<uint8_t> decompress_block(int kind, const uint8_t* in, size_t len, size_t expect);

uint64_t fnv1a64(const void* data, size_t n, uint64_t h = 0xCBF29CE484222325ull);

// Parsed fixed header of a container (include/dlmc.h describes the layout).
struct ContainerInfo {
  dlmc_codec_params cp{};
  uint64_t n = 0, n_chunks = 0, hash = 0, seed = 0;
  uint64_t first = 0, count = 0;  // held chunk range
  uint64_t total = 0;             // bytes of the (uncompressed) payload section
  uint32_t hdr = 0;               // header bytes before the payload section
};
void parse_header(const uint8_t* in, uint64_t len, ContainerInfo* ci);
std::vector<uint8_t> merge_containers(const uint8_t* const* parts, const uint64_t* lens, int n_parts);
uint64_t encode_bound(const dlmc_codec_params& cp, uint64_t n, uint64_t first, uint64_t count);
uint64_t numerics_id();
uint32_t crc32(const void* data, size_t n);
void create_model(dlmc_model* m, const dlmc_model_config& cfg, uint64_t seed, int device);
void validate_codec(const dlmc_model* m, const dlmc_codec_params& cp);

}  // namespace dlmc

struct dlmc_session {
  dlmc_model* m = nullptr;
  dlmc_codec_params cp{};
  bool encode = true;
  uint64_t n = 0;
  std::vector<int32_t> tokens;     // encode input / decode output
  std::vector<std::vector<uint8_t>> payload;  // per chunk (encode output / decode input)
  std::vector<uint32_t> crc;                  // per chunk (decode: expected)
  uint64_t n_chunks = 0, n_full = 0;
  uint64_t first_chunk = 0, end_chunk = 0;  // the chunk range [first, end) coded here
  int last_len = 0;

  // pass-loop state
  int phase = 0;  // 0: full-length chunks, 1: the final partial chunk, 2: done
  int B = 0, T = 0;
  uint64_t next_chunk = 0;
  std::vector<int64_t> slot_chunk;
  std::vector<int> slot_left, slot_pass;
  std::vector<dlmc::RangeEncoder> encs;
  std::vector<dlmc::RangeDecoder> decs;
  std::vector<dlmc::RansEncoder> rencs;
  std::vector<dlmc::RansDecoder> rdecs;
  // symbol ranking: per slot varint streams (encode output / decode input)
  std::vector<std::vector<uint8_t>> rk_out;
  std::vector<const uint8_t*> rk_data;
  std::vector<size_t> rk_len, rk_pos;
  std::vector<int32_t> rk_rank;  // decode: the ranks of the current pass (trace)
  // decode with the range coder or rANS: the payload section on the device,
  // each chunk's offset in it, and the slots' decoder states (device, and the
  // host copy of the last pass's)
  uint8_t* d_payload = nullptr;
  std::vector<uint64_t> pl_off;
  dlmc::DecSlot* d_dslot = nullptr;
  dlmc::DecSlot* h_dslot = nullptr;
  // initial context and left-to-right block schedules
  std::vector<std::vector<int32_t>> slot_ctx_pos, slot_ctx_sym;  // per slot
  std::vector<std::vector<int32_t>> slot_order;  // masked positions, ascending
  std::vector<int> slot_cursor;                  // next index into slot_order
  std::vector<int> blocks;                       // block sizes of the current phase
  bool started = false;
  uint64_t passes = 0;

  // pinned host staging
  int32_t* h_nsel = nullptr;
  int32_t* h_pos = nullptr;
  int32_t* h_err = nullptr;
  uint32_t* h_sym = nullptr;
  uint32_t* h_cdf = nullptr;  // trace only (allocated on first use): m_max * (V+1)
  int32_t* h_dec = nullptr;
  int64_t* h_base = nullptr;
  int32_t* h_state = nullptr;   // max_batch * max_chunk: a slot's initial state
  int32_t* h_rows = nullptr;    // block schedules: head rows, selections, counts
  int32_t* h_selpos = nullptr;
  int32_t* h_selrow = nullptr;
  int32_t* h_nsel_up = nullptr;

  ~dlmc_session();
  void begin_phase();
  void assign(int b, uint64_t chunk);
  int step(uint64_t* coded);  // returns 1 when done
  std::vector<uint8_t> container() const;
};
