// Host-side launchers of the gfx950 kernels (internal to the library).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lmop {

typedef uint16_t half_bits;  // fp16 storage as seen from host code

// ---------------------------------------------------------------- W4A16 GEMM
// Repacked int4 weight of one (possibly fused) linear map, N' x K':
//   qpack: u32 [Np/64][KG][64 lanes][4]; lane 16g+c, word f holds the 8 codes
//          of column nb*64 + 16f + c, features kg*32 + 8g .. +7, biased by +8,
//          nibble p = feature 2p (p < 4) / 2(p-4)+1 (p >= 4)
//   spack: fp16 [Np/64][KG][16 c][4 f]
// Np is a multiple of 256, Kp (= 32*KG) a multiple of 64.
// A linear map packed for the GEMM: int4 codes and fp16 group scales
// (spack), or FP8 codes and fp32 per-column scales (sscale).
struct PackedW {
  uint32_t* qpack = nullptr;
  half_bits* spack = nullptr;
  float* sscale = nullptr;
  int n = 0;   // logical output columns (fused)
  int np = 0;  // padded columns
  int kp = 0;  // padded input features (multiple of 64)
  int k = 0;   // logical input features
};

enum Epilogue : int {
  EPI_STORE_F16 = 0,  // C[m][n] = fp16(acc)
  EPI_ADD_F32 = 1,    // X[m][n] += acc (residual stream)
  EPI_SWIGLU = 2,     // fused [gate|up] blocks of 32: C[m][j] = fp16(silu(gate_j) * up_j)
  EPI_HEAD = 3,       // LM head (A = tiled head weight, B = hidden rows): per token and 128-entry
                      // vocabulary slice (max, sum exp), allowed-token logits, debug dump
  EPI_QKV = 4         // fused q|k|v: RoPE on q, k; q -> qout, k -> K store, v -> V^T store
};

struct GemmArgs {
  const void* A;  // fp16 [M][lda]; columns >= K are never read
  int lda;
  int M, N, K;    // N: columns of the (padded) weight walked by the grid; K multiple of 64
  // int4 weight (bq codes, bs fp16 group scales) or FP8 weight (bq E4M3
  // codes, bsc fp32 per-column scales)
  const uint32_t* bq;
  const half_bits* bs;
  const float* bsc;
  // fp16 weight (LM head): [N][ldb]
  const half_bits* bh;
  int ldb;
  // epilogue outputs
  void* C;        // fp16 [M][ldc]
  int ldc;
  int n_out;      // EPI_STORE_F16: valid columns; EPI_SWIGLU: output columns written
  float* X;       // fp32 [M][ldx]
  int ldx;
  // head epilogue (M = vocabulary, N = tokens)
  float2* part;          // [N][ceil(M/128)] (max, sum exp(z - max))
  const int32_t* sel;    // [M]: index of the vocabulary entry in the allowed list, or -1
  float* zsel;           // [N][n_sel]
  int n_sel;
  float* dump;           // NULL or fp32 [N][ld_dump]
  int ld_dump;
  // qkv epilogue.  Packed column order: q heads, k heads, v heads; every head
  // is hd/64 blocks of 64 columns; in a q/k block b of a head the columns are
  // dims [32b, 32b+32) then [hd/2 + 32b, hd/2 + 32b + 32), so each rotation
  // pair (d, d + hd/2) sits in one lane; v blocks keep the natural order.
  const int32_t* pos;    // [M] position of each token
  const int32_t* slot;   // [M] KV slot of each token
  const float2* rope;    // [max_seq][hd/2] (cos, sin)
  half_bits* qout;       // [M][nq*hd]
  half_bits* kc;         // layer's K store [cap][nkv][hd]
  half_bits* vt;         // layer's V^T store [nkv][hd][cap]
  int cap;
  int nq, nkv, hd;
};

// Picks the tile shape for M and launches.  Returns hipSuccess or the launch error.
hipError_t launch_gemm_w4(hipStream_t s, const GemmArgs& a, int epi);
hipError_t launch_gemm_w8(hipStream_t s, const GemmArgs& a, int epi);  // FP8 weights
hipError_t launch_gemm_f16(hipStream_t s, const GemmArgs& a, int epi);  // head only
// the head writes one (max, sum exp) partial per row and chunk of this many
// vocabulary entries, for any number of rows
constexpr int kHeadVocabChunk = 128;
// The LM head weight as the library keeps it: tiles of kHeadTileRows
// vocabulary rows x 32 features, [ceil(V / 128)][d / 32][128][32] fp16, rows
// past the vocabulary zero; tile (t, s) is 8 KB of contiguous memory.
constexpr int kHeadTileRows = 128;
// element (v, k) of the tiled head weight
__host__ __device__ inline size_t head_tiled_index(int v, int k, int d) {
  return (((size_t)(v / kHeadTileRows) * (d / 32) + k / 32) * kHeadTileRows + v % kHeadTileRows) *
             32 + k % 32;
}
// row-major fp16 [V][d] -> tiled (d a multiple of 32)
hipError_t launch_repack_head(hipStream_t s, const half_bits* src, int V, int d, half_bits* dst);

// Repacks one source matrix's rows into columns of a packed weight.
// colsrc[j] (device, [np]): (source index << 24) | source row, or -1 (zero column).
struct RepackSrc {
  const uint8_t* q[3];
  const half_bits* s[3];   // int4: fp16 group scales
  const float* sf[3];      // FP8: fp32 per-row scales
  int kp_src[3];  // int4: padded K of each source (multiple of 32); FP8: K
};
hipError_t launch_repack_w4(hipStream_t s, const RepackSrc& src, const int32_t* colsrc,
                            PackedW& dst);
// FP8 rows [n][K] of E4M3 codes -> tiles of 2 KB per 64 columns x 32
// features (two 1 KB halves; lane 16g+c of half h holds the 8 codes of
// features 8g.. of columns 16(2h)+c and 16(2h+1)+c), scales in column order
hipError_t launch_repack_w8(hipStream_t s, const RepackSrc& src, const int32_t* colsrc,
                            PackedW& dst);

// ---------------------------------------------------------------- elementwise
// p[i] = value for n_words 32-bit words (p 16-byte aligned)
hipError_t launch_fill_u32(hipStream_t s, void* p, size_t n_words, uint32_t value);
hipError_t launch_embed(hipStream_t s, const int32_t* tok, int T, const half_bits* emb, int d,
                        float* x);
// x_out[i] = x[idx[i]] (fp32, d), a_out[i] = a[idx[i]] (fp16, da)
hipError_t launch_gather_rows(hipStream_t s, const int32_t* idx, int R, const float* x, int d,
                              float* x_out, const half_bits* a, int da, half_bits* a_out);
// out[i] = fp16(rows[i] / rms(rows[i]) * gamma); rows[i] = x + i*ldx, or rowptr[i] if given
hipError_t launch_rmsnorm(hipStream_t s, const float* x, int ldx, const float* const* rowptr,
                          int R, const float* gamma, int d, float eps, half_bits* out, int ldo);

// ---------------------------------------------------------------- attention
// KV store of C slots (C a multiple of 64), per layer: K [C][nkv][hd] then
// V^T [nkv][hd][C]; layers follow each other ([L][2][C*nkv*hd]).
struct AttnRow {
  const half_bits* seg_kv[2];  // prefix-chain KV stores (root, child), or NULL
  int seg_n[2];                // tokens of each segment (0 if absent)
  int seg_cap[2];              // slots C of each segment's store
  int seg_start[2];            // slot of the segment's first token in its store
  int q_start;                 // first query token of the row in the batch buffers
  int n_q;                     // query tokens of the row in this launch
  int own_slot;                // slot of own token 0 in the own-KV store (multiple of 8)
  int own_q0;                  // own index of the first query token
};
constexpr int ATTN_QTILE = 128;  // query vectors (token, head-in-group) per workgroup
// Largest KV store (slots) the attention kernel reads: it forms V^T row
// offsets with a 24-bit multiply (dim x 2*capacity bytes).
constexpr int kMaxStoreSlots = 1 << 22;

struct AttnArgs {
  const half_bits* q;  // [T][ldq], post-RoPE
  int ldq;
  half_bits* out;      // [T][ldo]
  int ldo;
  const AttnRow* rows;
  const int2* work;    // (row, ATTN_QTILE-query tile)
  int n_work;
  const half_bits* own_kv;  // own-KV store, own_cap slots
  int own_cap;
  int layer;
  int nq, nkv, hd;
};
hipError_t launch_attention(hipStream_t s, const AttnArgs& a);

// ---------------------------------------------------------------- head finalize
struct HeadPick {
  int32_t index;   // position in the allowed list
  int32_t token;
  float logprob;   // over the allowed set
  float logprob_full;
  float margin;    // top-two allowed gap
  float pad[3];
};
// per row: combine partials -> LSE over V; pick among zsel[:n_allowed]
// zsel[r][i] = hn[r] . W[allowed[i]] (W the tiled head weight, fp32 sums)
// for the n_sel allowed tokens only; with dump, also dump[r][allowed[i]]
hipError_t launch_head_restricted(hipStream_t s, const half_bits* hn, int R, int d,
                                  const half_bits* W, const int32_t* allowed, int n_sel,
                                  float* zsel, float* dump, int ld_dump);
// n_chunks = 0: no vocabulary partials (restricted head), logprob_full = NaN.
// state_mask != NULL: row r picks only among entries j < n_allowed with
// state_mask[row_state[r] * n_sel + j] != 0 (token-automaton outputs).
hipError_t launch_head_finalize(hipStream_t s, const float2* part, int n_chunks,
                                const float* zsel, int n_sel, int n_allowed,
                                const int32_t* allowed_tok, int R, HeadPick* out,
                                const int32_t* row_state = nullptr,
                                const uint8_t* state_mask = nullptr);

}  // namespace lmop
