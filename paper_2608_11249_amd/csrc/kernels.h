// Host-side launchers of the HIP kernels of the masked-diffusion step.
#pragma once

#include "common.h"

namespace dlmc {

// ---------------------------------------------------------------- GEMMs
// Epilogues fused into C = A * B^T (A [M, K] activations, B [N, K] weights).
enum EpiKind : int {
  EPI_STORE_F32 = 0,  // out_f32[row * ldo + col] = acc                 (LM head logits)
  EPI_RESIDUAL = 1,   // x[row * ldo + col] += acc                      (O-proj, FFN out)
  EPI_QKV_ROPE = 2,   // Q, K with rotary embedding, V transposed       (QKV projection)
  EPI_GELU = 3,       // out_bf16[row * ldo + col] = gelu(acc)          (FFN in, GELU)
  EPI_SWIGLU = 4,     // out_bf16[row * ldo + col/2..] = silu(g) * u     (FFN gate/up pairs)
};

struct EpiArgs {
  void* out = nullptr;  // float* or bf16_t* depending on the epilogue
  int ldo = 0;
  // EPI_QKV_ROPE: Q, K are [B, H, Tp, dh]; Vt is [B, H, dh, Tp]
  void* q = nullptr;
  void* k = nullptr;
  void* vt = nullptr;
  const float* rope_cos = nullptr;  // [T, dh/2]
  const float* rope_sin = nullptr;
  int T = 0, Tp = 0, H = 0, dh = 0, d = 0;
  // EPI_STORE_F32 (optional): softmax statistics of every 128-column group of
  // every stored row, RowStat [rows, stat_ld] (rowstats.h)
  void* stats = nullptr;
  int stat_ld = 0;
};

// Tile shape of a bf16 GEMM (the choice never changes the result):
// 128 x 128 or 192 x 128 tiles two blocks per CU, or the 4-wave kernel with
// columns [0, split) on 256 x 256 tiles and [split, N) on 256 x 128 tiles.
enum GemmTileKind { GEMM_TILES_128x128 = 0, GEMM_TILES_192x128 = 1, GEMM_TILES_4WAVE = 2 };
struct GemmTiles {
  int kind, split;
};
// the choice gemm_bf16 makes for these sizes (d: the QKV epilogue's model
// width); host only
GemmTiles gemm_bf16_tiles(int M, int N, int K, EpiKind epi, int d, int rows_hint);
// M_dev (optional): device int holding the live row count (<= M); rows at or
// beyond it are neither computed (whole tiles) nor stored.  rows_hint: the
// live row count if the host knows it (tile selection only), else -1.
void gemm_bf16(hipStream_t st, const bf16_t* A, const bf16_t* B, int M, int N, int K,
               const int* M_dev, EpiKind epi, const EpiArgs& ea, int rows_hint = -1);
void gemm_f32(hipStream_t st, const float* A, const float* B, int M, int N, int K,
              const int* M_dev, EpiKind epi, const EpiArgs& ea);

// fp32 path helpers (the bf16 path fuses these into GEMM epilogues)
void qkv_rope_f32(hipStream_t st, const float* qkv, int M, const EpiArgs& ea);
void ffn_act_f32(hipStream_t st, const float* in, float* out, int M, int F, int kind);

// ---------------------------------------------------------------- attention
// Non-causal softmax(Q K^T / sqrt(dh)) V over all T keys of each chunk.
// out is [B*T, H*dh] row-major.
void attention_bf16(hipStream_t st, const bf16_t* q, const bf16_t* k, const bf16_t* vt,
                    bf16_t* out, int B, int H, int T, int Tp, int dh);
void attention_f32(hipStream_t st, const float* q, const float* k, const float* vt, float* out,
                   int B, int H, int T, int Tp, int dh);

// ---------------------------------------------------------------- elementwise
// Row layout of an initialised weight tensor inside its device buffer.
enum RowMap : int {
  MAP_IDENTITY = 0,  // device row = canonical row + offset
  MAP_QK_PAIRS = 1,  // rotate-half pairs (i, i + dh/2) moved to adjacent 32-row blocks
  MAP_GLU_PAIRS = 2, // gate/up features interleaved in 32-row blocks (up: offset 32)
};
void init_weights(hipStream_t st, void* dst, int dtype, uint64_t seed, int tensor_id, int rows,
                  int cols, int exp, RowMap map, int row_offset, int dh);
void embed(hipStream_t st, const int32_t* state, const void* table, int dtype, float* x,
           int n_rows, int d, int max_id);
// gather_rows (optional): output row i normalises x[gather_rows[i]]; n_dev
// (optional) holds the live row count.
void norm_rows(hipStream_t st, const float* x, void* out, int out_dtype, int n_rows, int d,
               int norm_kind, float eps, const int32_t* gather_rows, const int32_t* n_dev);
void fill_i32(hipStream_t st, int32_t* p, int32_t v, size_t n);
// dst[b*m_max + j] = src[sel_row[b*m_max + j]] (rows of d bf16) and
// dst_mx[b*m_max + j] = mx[sel_row[b*m_max + j]] for j < n_sel[b], else zeros
void gather_slot_rows(hipStream_t st, const bf16_t* src, const float* mx, const int32_t* sel_row,
                      const int32_t* n_sel, int B, int m_max, int d, bf16_t* dst, float* dst_mx);

// ---------------------------------------------------------------- coding stages
// rows[] = flat indices b*T+t with state == mask_id (ascending), n_rows[0],
// chunk_off[b] / chunk_cnt[b] = the segment of chunk b inside rows[].
void compact_masked(hipStream_t st, const int32_t* state, int B, int T, int mask_id,
                    int32_t* rows, int32_t* n_rows, int32_t* chunk_off, int32_t* chunk_cnt);
// per row of logits[n, V]: entropy in bits and row max (n from n_dev when given)
void entropy_rows(hipStream_t st, const float* logits, int n_max, const int32_t* n_dev, int V,
                  float* H, float* mx);
// the same from the 128-column group statistics the LM head's epilogue
// wrote (stats: RowStat [n, ld]); bit-identical to entropy_rows
void entropy_merge(hipStream_t st, const void* stats, int ld, int V, int n_max, const int32_t* n_dev,
                   float* H, float* mx);
// commitment schedule, one workgroup per chunk
void select_positions(hipStream_t st, const float* H, const int32_t* rows,
                      const int32_t* chunk_off, const int32_t* chunk_cnt, int B, int T,
                      float tau, int m_min, int m_max, int32_t* sel_pos, int32_t* sel_row,
                      int32_t* n_sel, int32_t* err_flag);
// integer CDF of row sel_row[b*m_max+j] of logits (for j < n_sel[b]) into
// cdf[(b*m_max+j)*(V+1) ..]; g_out (optional) receives the g values.
// seg_ws: device workspace of cdf_workspace_bytes(B * m_max, V) bytes.
int cdf_segments(int V);
inline size_t cdf_workspace_bytes(size_t slots, int V) {
  return slots * (size_t)cdf_segments(V) * (8 + 8 + 4);
}
void cdf_rows(hipStream_t st, const float* logits, const float* mx, const int32_t* sel_row,
              const int32_t* n_sel, int B, int m_max, int V, int P, uint32_t* cdf,
              uint32_t* g_out, void* seg_ws);
// ---------------------------------------------------------------- static scratch
// Bytes of the static device scratch used by the allocation-free entry point.
constexpr size_t SCRATCH_BYTES = DLMC_SCRATCH_BYTES;
// Device address of `device`'s copy of the scratch (looked up on first use,
// with that device current; each GPU holds its own copy).
void* scratch_address(int device);
// sel_row[i] = i, n_sel[i] = 1 for i < n (one committed row per "chunk")
void fill_row_slots(hipStream_t st, int32_t* sel_row, int32_t* n_sel, int n);

// test hook: a NaN into element 0 of the head's input rows (bf16 or fp32)
// when n_dev[0] > 0, which makes the first head row non-finite
void poison_head_input(hipStream_t st, void* rows, int bf16, const int32_t* n_dev);
// encode: (start, freq) of the true symbol of every committed position and reveal it
void gather_reveal(hipStream_t st, const uint32_t* cdf, const int32_t* sel_pos,
                   const int32_t* n_sel, const int32_t* tokens, const int64_t* slot_base,
                   int32_t* state, int B, int T, int m_max, int V, uint32_t* sym);
// decode: reveal decoded symbols
void reveal(hipStream_t st, const int32_t* sel_pos, const int32_t* n_sel, const int32_t* dec,
            int32_t* state, int B, int T, int m_max);
// decode: the entropy decoder of one batch slot, kept in device memory between
// passes.  Range coder: x = code - low and range; rANS: x = the state.  pos /
// len: read position and length (bytes) of the slot's stream, which starts at
// byte off of the payload buffer.  Slots with live = 0 decode nothing.
struct DecSlot {
  uint64_t x, range, pos, len, off;
  uint32_t live, pad;
};
// decode: one wave per live slot b decodes the slot's n_sel[b] committed
// symbols of the pass, in slot order, from CDF rows b * m_max + j (V + 1 words
// each) with the arithmetic of the host decoders (W-bit range coder, or rANS
// with lower bound rans_lo when `rans`); writes dec[slot] = symbol and
// iv[2 slot], iv[2 slot + 1] = (start, freq), and the slot's new state.  A
// corrupt stream stops its slot and sets *err to 2 if it was 0.
void decode_symbols(hipStream_t st, const uint32_t* cdf, const int32_t* n_sel, int B, int m_max,
                    int V, int P, int W, bool rans, uint64_t rans_lo, const uint8_t* payload,
                    DecSlot* slots, int32_t* dec, uint32_t* iv, int32_t* err);
// attention-based context: A[i, :] (+)= w softmax(scale S[i, :]) (rows T,
// pitch T), and out = (A^T v + v) / 2
void softmax_accumulate(hipStream_t st, const float* S, float* A, int T, float scale, float w,
                        bool first);
void rollout_step(hipStream_t st, const float* A, const float* v, float* out, int T);
// symbol ranking: encode writes (rank, symbol) pairs to out[2 * slot], decode
// turns the ranks in dec[slot] into symbols; both reveal the symbols in state
void rank_symbols(hipStream_t st, const float* logits, const int32_t* sel_row,
                  const int32_t* sel_pos, const int32_t* n_sel, const int32_t* tokens,
                  const int64_t* slot_base, int32_t* state, int B, int T, int m_max, int V,
                  uint32_t* out);
void select_by_rank(hipStream_t st, const float* logits, const int32_t* sel_row,
                    const int32_t* sel_pos, const int32_t* n_sel, int32_t* dec, int32_t* state,
                    int B, int T, int m_max, int V);

}  // namespace dlmc
