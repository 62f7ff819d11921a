// internal.hpp -- host-side interface between the C-ABI layer (api.hip) and
// the kernel launchers (kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "device.hpp"

namespace nmt {

constexpr int kMaxTpad = 1024;     // attention keeps one score per source position in LDS
// Launch shapes that depend on how many blocks fill the chip take the
// device's compute-unit count (read once per model; 256 on MI355X, in 8
// XCDs of 32) as an argument named `cus`.

// K chunk of the GEMM tiles: 8 sixteen-byte vectors of 4 fp32 or 8 bf16.
inline int chunk_k(bool bf16) { return bf16 ? PrecBF16::KC : PrecF32::KC; }

// Tile shapes (rows x packed columns) of the kernel families.
constexpr int kPlainSmallTM = 64, kPlainSmallTN = 64;    // 4 waves of 32 x 32
constexpr int kPlainLargeTM = 128, kPlainLargeTN = 128;  // 4 waves of 64 x 64
// GRU tile: TM rows x HB hidden units (3*HB packed columns), waves of WM rows
// x 32 units.  Overridable at compile time for tuning sweeps.
#ifndef NMT_GRU_TM
#define NMT_GRU_TM 128
#endif
#ifndef NMT_GRU_WM
#define NMT_GRU_WM 32
#endif
#ifndef NMT_GRU_TM_BF16
#define NMT_GRU_TM_BF16 128
#endif
#ifndef NMT_GRU_HB_BF16
#define NMT_GRU_HB_BF16 64
#endif
#ifndef NMT_GRU_WM_BF16
#define NMT_GRU_WM_BF16 32
#endif
constexpr int kGruTM = NMT_GRU_TM, kGruHB = 64, kGruWM = NMT_GRU_WM;
constexpr int kGruTM16 = NMT_GRU_TM_BF16, kGruHB16 = NMT_GRU_HB_BF16, kGruWM16 = NMT_GRU_WM_BF16;  // bf16 weights
inline int gru_hb(bool bf16) { return bf16 ? kGruHB16 : kGruHB; }
// Rows of the GRU tile for small batches, used when the large tile would
// give fewer blocks than there are compute units.
#ifndef NMT_GRU_SMALL_TM
#define NMT_GRU_SMALL_TM 64
#endif
constexpr int kGruSmallTM = NMT_GRU_SMALL_TM;
// Which kernel form the bf16 GRU and small-tile plain products take: 0 the
// weight-streaming one where it applies and fills the chip, 1 wherever it
// applies, 2 never, 3 and 4 as 1 with the plain products' in-block K split
// off or on (a test switch, set through nmt_debug_gemm_form).
extern std::atomic<int> g_gemm_form;
inline bool gemm_stream_forced(int form) { return form == 1 || form == 3 || form == 4; }
extern std::atomic<int64_t> g_gemm_streamed;  // launches of the weight-streaming form
constexpr int kVocabTN = 32;                    // packing granularity of the output weights
constexpr int kVocabSpare = 32;                 // zero columns past the last block (group loads stay inside)

// A weight matrix packed for one kernel family: [Kpad/KV][Npad][KV] of fp32
// (KV = 4) or bf16 (KV = 8), 16 bytes per (vector row, column).
struct Packed {
  void* d = nullptr;
  bool bf16 = false;
  int64_t Kpad = 0;  // sum of the padded K of its segments
  int64_t Npad = 0;
  int N = 0;         // valid columns (for GRU: 3H)
  // Output weights only: rows Krows .. Krows+nbias-1 of the packed matrix
  // hold the bias (fp32: one row; bf16: hi, mid, lo parts summing to it).
  int Krows = 0;
  int nbias = 0;
};

enum class Tile { Small, Large };
inline int tile_m(Tile t) { return t == Tile::Small ? kPlainSmallTM : kPlainLargeTM; }
inline int tile_n(Tile t) { return t == Tile::Small ? kPlainSmallTN : kPlainLargeTN; }

// Epilogue of the plain GEMM: out = act(acc + bias); rows with
// (m % mask_T) >= mask_len[m / mask_T] are written as zeros.  With
// ksplit > 1 the K chunks are split over ksplit blocks, which write raw sums
// to part [ksplit][M][N]; a reduce kernel then adds them in a fixed order
// and applies the epilogue (deterministic, no atomics).
struct PlainEpi {
  float* out;
  int64_t ldo;
  const float* bias;  // [N]
  int N;
  int act;            // 0: identity, 1: tanh
  const int32_t* mask_len;
  int32_t mask_T;
  int32_t ksplit = 1;
  float* part = nullptr;
  __bf16* out16 = nullptr;  // nullable: the output goes here in bf16 (nearest even) instead of to out
  int32_t defer_reduce = 0;  // ksplit > 1: leave the raw sums in part for the consumer to add (no epilogue)
  // nullable: row m's sums also get row add_row[m] of `add` (row stride
  // ld_add; rows outside [0, add_rows) add nothing), before bias and activation
  const float* add = nullptr;
  int64_t ld_add = 0;
  const int32_t* add_row = nullptr;
  int32_t add_rows = 0;
  // nullable: row m's sums also get row m of add2 (row stride ld_add2)
  const float* add2 = nullptr;
  int64_t ld_add2 = 0;
};

// Epilogue of the GRU gate GEMM (see device.hpp for the cell).
struct GruEpi {
  const float* h;     // previous state rows (nullable: zero state)
  int64_t ldh;
  const int32_t* hrow;  // nullable: row m's state is row hrow[m] of h (outside [0, hrows): zero state)
  int32_t hrows;
  const float* xin;   // nullable: precomputed input-side pre-activations [r|z|n] per row
  int64_t ldx;
  const float* brz;   // [2H] summed r,z biases
  const float* bni;   // [H] input-side candidate bias
  const float* bns;   // [H] state-side candidate bias (inside the reset gate)
  float* out;
  int64_t ldo;
  const int32_t* mask_len;  // nullable: row m is kept iff mask_pos < mask_len[m]
  int32_t mask_pos;
  int32_t H;
  __bf16* out16 = nullptr;  // nullable: a bf16 copy of out (nearest even), row stride ldo
  // nullable: row m's input-side pre-activations are row xrow[m] of xin
  // (rows outside [0, xrows): zeros)
  const int32_t* xrow = nullptr;
  int32_t xrows = 0;
};

struct GruProblem {
  AOperand A;
  const void* Wp;
  int64_t Npad;
  GruEpi ep;
};

// Launchers (all asynchronous on `st`).
// cus > 0 lets a small-tile bf16 product take the weight-streaming form.
hipError_t launch_gemm_plain(Tile t, const AOperand& A, const Packed& W, const PlainEpi& ep, hipStream_t st,
                             int cus = 0);
hipError_t launch_gemm_gru(const GruProblem* probs, int nprob, int H, bool bf16, int cus, hipStream_t st);
// K splits for a GRU launch of M rows whose A operand has `nchunks` K chunks:
// 1 when the launch fills the chip as it is, else enough splits of the tile
// gru_split_tm picks for about two 4-wave blocks (64 rows) or one 8-wave
// block (128 rows) per compute unit (each split at least four chunks, at
// most 8 splits).  Its launch needs part [ksplit][M][4][H].
int gru_ksplit(int M, int H, int nchunks, bool bf16, int cus);
// Rows of a split launch's tile: 128 where those tiles alone give half the
// CUs a block (so two splits fill the chip), else 64.
int gru_split_tm(int M, int H, bool bf16, int cus);
// The same with the K chunks split over ksplit blocks per tile: raw sums go
// to part [nprob][ksplit][part_M][4][H] (part_M >= every problem's rows), a
// second kernel adds them in split order and applies the cell.
hipError_t launch_gemm_gru_split(const GruProblem* probs, int nprob, int H, bool bf16, int ksplit, float* part,
                                 int part_M, int tm, hipStream_t st);
// Number of vocabulary slices (partials per row) for M rows, and the
// largest padded E the vocabulary kernel keeps in LDS.
int vocab_tm(int M, int V, bool bf16, int64_t Kpad, int E, int nb, int cus);
int vocab_slices(int M, int V, bool bf16, int cus, int tm);
int vocab_max_kpad(bool bf16);
bool vocab_offsets_fit(int64_t Kpad, int64_t Npad, bool bf16);
// Row stride of a bf16 copy of rows E wide: whole 16-byte vectors.
inline __host__ __device__ int bf16_row(int E) { return (E + 7) / 8 * 8; }
// t16: t is stored in bf16 (row stride bf16_row(E)) instead of fp32; the
// kernels never use the padding slots' contents (with_bias_ones).
// req1 (nullable): the requested words, one per row (req_off NULL) or CSR
// (req_off [M+1] over nreq words); the logit of each row that requests
// exactly one word goes to zreq [M] (rows whose word is outside [0, V), or
// whose span is malformed, get nothing written).  nS and tm: the slices and
// the row tile chosen for M rows by vocab_slices and vocab_tm.
hipError_t launch_vocab_lse(const float* t, int t16, int M, int E, const Packed& W, int V, float2* part, int nS,
                            int tm, const int32_t* req1, const int32_t* req_off, int nreq, float* zreq,
                            hipStream_t st);
// Requests of row b: req[req_off[b] .. req_off[b+1]) with logp at the same
// indices (req_off nullable: one request per row, req[b] -> logp[b]).  The
// combine takes the logits of rows with one request from zreq (the
// vocabulary kernel's, nullable) and scores the other rows' words with dot
// products of their own.
// state_row (nullable) is checked against pool_rows like the other ids.
struct Requests {
  const int32_t* req_off;
  const int32_t* req;
  int32_t nreq;
  const int32_t* state_row;
  int32_t pool_rows;
};
hipError_t launch_lse_combine(int B, const float2* part, int nS, const float* t, int t16, int E, const Packed& W, int V,
                              const Requests& rq, const int32_t* y_prev,
                              const int32_t* sent_id, int S, float* logp, float* logZ, int* err,
                              const float* zreq, hipStream_t st);
// Attention groups rows by sentence through workspace arrays: perm [B]
// int32, tiles [B] int4, n_tiles [1] int32 (perm NULL: one block per row).
constexpr int kGroupMaxS = 8192;  // sentences the grouping kernel can count in LDS
constexpr int kAttnGroup = 4;  // rows per attention tile (fewer when the tiles would not cover the CUs)
#ifndef NMT_ATTN_WAVES
#define NMT_ATTN_WAVES 8
#endif
constexpr int kAttnWaves = NMT_ATTN_WAVES;
constexpr int kAttnWideTiles = 640;  // grouped-attention launches of at most this many blocks use 2 * kAttnWaves waves
#ifndef NMT_ATTN_CU
#define NMT_ATTN_CU 4
#endif
#ifndef NMT_ATTN_SNAKE
#define NMT_ATTN_SNAKE 1
#endif
struct AttnGroups {
  int32_t* perm;
  int4* tiles;
  int32_t* n_tiles;
  int32_t one_sentence = -1;  // >= 0: every row is this sentence, tiled in row order with no grouping
};
// kfac [S x Tpad x A]: the keys' factors 2^{2 log2(e) pctx}, kbig [S] the
// sentences whose keys are too large for them (launch_key_factors); pctx the
// keys themselves, which tiles with such keys and large queries score from.
// c_bf16: the context c [B x C] is written in bf16 (nearest even) instead of fp32.
// The attention's queries: q [B x A], or (ks > 1) the query GEMM's unreduced
// split-K sums, ks blocks of `stride` floats laid out like q, which the
// attention adds in split order as it loads them (the GEMM's own reduction,
// without its launch).
struct QuerySrc {
  const float* q;
  int32_t ks;
  int64_t stride;
};
__device__ __forceinline__ f32x4 load_q(const QuerySrc& q, int row, int A, int a4) {
  const float* p = q.q + (int64_t)row * A + 4 * a4;
  if (q.ks <= 1) return *(const f32x4*)p;
  f32x4 v = zero4();
  for (int z = 0; z < q.ks; ++z) v += *(const f32x4*)(p + z * q.stride);
  return v;
}
// grouped: grp already holds this batch's grouping (launch_group_levels, with
// G = attn_rows_per_tile(B, cus)), so no grouping kernel runs.
hipError_t launch_attention(int B, int A, int C, int Tpad, QuerySrc q, const float* kfac, const float* pctx,
                            const int32_t* kbig, const float* ctx, const int32_t* len, const int32_t* sent_id, int S,
                            const float* v, float* c, float* alpha, const AttnGroups& grp, bool c_bf16,
                            int cus, hipStream_t st, bool grouped = false);
// Rows per attention tile for a batch of B rows: kAttnGroup, halved while the
// tiles would leave more than half the CUs idle.
int attn_rows_per_tile(int B, int cus);
// The grouping of several batches (the levels of a forest) in one launch,
// one block per batch: rows B of sentences sent_id, tiles of G rows.
struct GroupLevel {
  int32_t B, G;
  const int32_t* sent_id;
  AttnGroups grp;
};
constexpr int kMaxGroupLevels = 16;  // batches per launch
hipError_t launch_group_levels(const GroupLevel* lv, int n, int S, const int32_t* len, int Tpad, hipStream_t st);
hipError_t launch_bf16_to_f32(const void* x, int64_t rows, int cols, int64_t ld, float* y, hipStream_t st);
// Per sentence of the keys pctx [S x Tpad x A] (A a multiple of 4):
// kfac = 2^{2 log2(e) pctx}, exponent clamped to [-126, 126], and big[s] = 1
// when some exponent of sentence s exceeds the range where the clamped
// factors still score exactly (0 otherwise).
hipError_t launch_key_factors(int S, int Tpad, int A, const float* pctx, float* kfac, int32_t* big, hipStream_t st);
hipError_t launch_check_src_ids(int S, int Tpad, const int32_t* ids, const int32_t* len, int V_src,
                                int* err, hipStream_t st);
hipError_t launch_masked_copy(int S, int Tpad, int C, const float* src, const int32_t* len, float* dst,
                              hipStream_t st);
hipError_t launch_masked_mean(int S, int Tpad, int C, const float* ctx, const int32_t* len, float* mean,
                              hipStream_t st);

// Several models at once: buffer pointers and weights, passed by value.
constexpr int kMaxModels = 32;
struct ModelTable {
  const void* p[kMaxModels];
  float w[kMaxModels];
};
// kind 1: fp32 buffer, 2: bf16 buffer; round_bf16 rounds fp32 results to bf16 values.
hipError_t launch_average(int K, int64_t n, const ModelTable& tab, int kind, bool round_bf16, void* dst,
                          hipStream_t st);
hipError_t launch_weighted_sum(int K, int B, const float* logp, const ModelTable& tab, float* out, hipStream_t st);

// Every device allocation and release of the library (the test hook of
// nmt_debug.h can make allocations fail, and counts live ones).
hipError_t device_malloc(void** p, size_t bytes);
void device_free(void* p);

inline int ceil_div(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }
inline int64_t round_up(int64_t a, int64_t b) { return (a + b - 1) / b * b; }

}  // namespace nmt
