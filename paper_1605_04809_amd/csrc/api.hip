// api.hip -- the C-ABI of libnmt (declared in include/nmt.h): model upload
// and re-layout, source initialisation, and the batched decoder step
// (Section 5.1 of the paper: NMT(H_{i-1}, E_i) over a precomputed source
// context).  Every arithmetic step runs in the kernels of kernels.hip; this
// file validates arguments, packs weights once, and enqueues launches.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <cmath>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include "../../include/nmt.h"
#include "../../include/nmt_debug.h"
#include "../../include/nmt_profile.h"
#include "internal.hpp"

using namespace nmt;

namespace {

thread_local std::string g_err;

// The allocation test hook (nmt_debug.h): allocations left before injected
// failures (-1: none), and the library's live device allocations.
std::atomic<int64_t> g_alloc_budget{-1};
std::atomic<int64_t> g_live_allocs{0};
std::atomic<int32_t> g_precompute{1};  // nmt_debug_precompute

nmt_status fail(nmt_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

nmt_status ok() {
  g_err.clear();
  return NMT_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// Device allocations owned by a model or a source.
// A model's parameter buffers are tagged so that nmt_model_average can walk
// them without knowing what each one holds.
enum AllocKind : uint8_t { kOther = 0, kParamF32 = 1, kParamBF16 = 2 };

struct Allocs {
  std::vector<void*> ptrs;
  std::vector<size_t> bytes;
  std::vector<uint8_t> kind;
  hipError_t alloc(void** p, size_t n, uint8_t k = kOther) {
    hipError_t e = device_malloc(p, n < 256 ? 256 : n);
    if (e == hipSuccess) {
      ptrs.push_back(*p);
      bytes.push_back(n);
      kind.push_back(k);
    }
    return e;
  }
  void release() {
    for (void* p : ptrs) device_free(p);
    ptrs.clear();
    bytes.clear();
    kind.clear();
  }
};

struct GruBias {
  float *brz = nullptr, *bni = nullptr, *bns = nullptr;
};

}  // namespace

struct nmt_model {
  nmt_dims dims{};
  int device = 0;
  int cus = 0;        // the device's compute units (launch shapes that fill the chip)
  bool bf16 = false;  // weights and embeddings stored as bf16
  int kc = 32;        // K chunk of the GEMM tiles
  int64_t emb_ld = 0; // row stride of the embedding tables (elements)
  Allocs mem;
  void *emb_src = nullptr, *emb_tgt = nullptr;
  Packed enc_in, enc_U[2], att_Wc, init_W, g1, att_Wq, g2, ro, out;
  // precomp (fp32 weights): the products of the previous word's embedding
  // (the first GRU's input side and the readout's word term) are per-word
  // tables [V x 3H] and [V x E], built from the embedding table and the
  // packed weights g1x and roy when the model is created (or averaged), and
  // the products of the context (the second GRU's input side and the
  // readout's context term) are mixed by the attention from per-position
  // projections of the annotations, [S x Tpad x cpw_ld], made with cpw when
  // a source is set up; g1, g2 and ro then hold only the state-side
  // weights.  bf16 weights keep all these products in the step: their GEMMs
  // are bound by memory traffic, which fp32 table rows and projections
  // would raise.
  bool precomp = false;
  Packed g1x, roy, cpw;
  int cpw_ld = 0;  // columns of a projection row: 3H + E, padded to the large tile
  float *tab_x = nullptr, *tab_y = nullptr;
  float *enc_in_b = nullptr, *att_b = nullptr, *init_b = nullptr, *att_v = nullptr, *ro_b = nullptr;
  GruBias enc_bias, g1_bias, g2_bias;
  int* err = nullptr;  // sticky device error flag
  void* noalloc_ws = nullptr;  // this device's copy of the allocation-free step's scratch array
  // event timing of the step's phases (nmt_profile.h); not thread-safe
  std::vector<hipEvent_t> prof_events;  // (NMT_NUM_PHASES + 1) per timed step
  int prof_max = 0, prof_used = 0;
  bool prof_on = false;
};

struct nmt_source {
  int32_t S = 0, Tpad = 0;
  int32_t H = 0, A = 0, cpw_ld = 0;  // the widths of the model that set it up
  Allocs mem;
  float *ctx = nullptr, *pctx = nullptr, *scratch = nullptr;
  float* kfac = nullptr;  // 2^{2 log2(e) pctx}: the keys' factors of the attention scores
  // precomp models: per position, the annotation times the second GRU's
  // input-side weights [r | z | n] and the readout's context weights, then
  // zeros to cpw_ld columns
  float* cproj = nullptr;
  int32_t* kbig = nullptr;  // [S] 1 where a sentence has keys too large for their factors
  float* gru_part = nullptr;  // encoder: the recurrent GRU's split-K sums [2][enc_ks][S][4H]
  int enc_ks = 1;
  int32_t* len = nullptr;
  std::vector<int32_t> h_len;
};

namespace {

// Host-side packing of x.W-oriented weights into the [Kpad/KV][Npad][KV]
// layout of the GEMM kernels (KV = 4 fp32 or 8 bf16).  Segments are stacked
// along K, each padded to a multiple of the chunk `kc`; `colmap(np)` gives
// the source column of packed column np (or -1 for a zero column).
struct Seg {
  const float* W;  // [K x ld] row-major
  int K;
  int ld;
  const float* X = nullptr;  // nullable: nx more rows [nx x ld] appended after the K rows of W
  int nx = 0;
};

uint16_t to_bf16(float x) {  // nearest, ties to even (inputs are finite)
  uint32_t u;
  memcpy(&u, &x, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

float bf16_value(float x) {  // x rounded to the nearest bf16 value, as fp32
  const uint32_t u = (uint32_t)to_bf16(x) << 16;
  float y;
  memcpy(&y, &u, 4);
  return y;
}

// Number of bias rows appended to the packed output weights: fp32 stores
// the bias in one row; bf16 in three (hi, mid, lo), whose exact sum is the
// fp32 bias, so the MFMA adds the same bias the fp32 path does.
int vocab_bias_rows(bool bf16) { return bf16 ? 3 : 1; }

template <class ColMap>
std::vector<float> pack_host(const std::vector<Seg>& segs, int64_t Npad, int kc, int KV, ColMap colmap,
                             int64_t* Kpad_out) {
  int64_t Kpad = 0;
  for (const Seg& s : segs) Kpad += round_up(s.K + s.nx, kc);
  std::vector<float> out((size_t)(Kpad * Npad), 0.f);
  std::vector<int> cols((size_t)Npad);
  for (int64_t np = 0; np < Npad; ++np) cols[(size_t)np] = colmap(np);
  int64_t koff = 0;
  for (const Seg& s : segs) {
    for (int k = 0; k < s.K + s.nx; ++k) {
      const int64_t kk = koff + k;
      float* dst = out.data() + (kk / KV) * Npad * KV + (kk % KV);
      const float* src = k < s.K ? s.W + (int64_t)k * s.ld : s.X + (int64_t)(k - s.K) * s.ld;
      for (int64_t np = 0; np < Npad; ++np) {
        const int c = cols[(size_t)np];
        if (c >= 0) dst[np * KV] = src[c];
      }
    }
    koff += round_up(s.K + s.nx, kc);
  }
  *Kpad_out = Kpad;
  return out;
}

hipError_t upload(Allocs& mem, float** d, const float* h, size_t n) {
  hipError_t e = mem.alloc((void**)d, n * sizeof(float), kParamF32);
  if (e != hipSuccess) return e;
  return hipMemcpy(*d, h, n * sizeof(float), hipMemcpyHostToDevice);
}

// Upload fp32 values as fp32 or (rounded) bf16.
hipError_t upload_w(Allocs& mem, void** d, const std::vector<float>& h, bool bf16) {
  if (!bf16) return upload(mem, (float**)d, h.data(), h.size());
  std::vector<uint16_t> b(h.size());
  for (size_t i = 0; i < h.size(); ++i) b[i] = to_bf16(h[i]);
  hipError_t e = mem.alloc(d, b.size() * 2, kParamBF16);
  if (e != hipSuccess) return e;
  return hipMemcpy(*d, b.data(), b.size() * 2, hipMemcpyHostToDevice);
}

// An embedding table [rows x E]: fp32 as is, bf16 with rows padded to `ld`.
hipError_t upload_table(Allocs& mem, void** d, const float* h, int64_t rows, int E, int64_t ld, bool bf16) {
  if (!bf16) return upload(mem, (float**)d, h, (size_t)rows * E);
  std::vector<float> padded((size_t)(rows * ld), 0.f);
  for (int64_t r = 0; r < rows; ++r) memcpy(&padded[(size_t)(r * ld)], h + r * E, sizeof(float) * E);
  return upload_w(mem, d, padded, true);
}

hipError_t pack_plain(Allocs& mem, Packed* P, const std::vector<Seg>& segs, int N, int TN, int kc, bool bf16,
                      int spare = 0) {
  P->N = N;
  P->bf16 = bf16;
  P->Npad = round_up(N, TN) + spare;
  std::vector<float> h =
      pack_host(segs, P->Npad, kc, bf16 ? 8 : 4, [N](int64_t np) { return np < N ? (int)np : -1; }, &P->Kpad);
  return upload_w(mem, &P->d, h, bf16);
}

// GRU packing: column tile u holds [r | z | n] of hidden units u*HB .. u*HB+HB-1.
hipError_t pack_gru(Allocs& mem, Packed* P, const std::vector<Seg>& segs, int H, int kc, bool bf16) {
  P->N = 3 * H;
  P->bf16 = bf16;
  const int HB = gru_hb(bf16);
  P->Npad = (int64_t)ceil_div(H, HB) * 3 * HB;
  std::vector<float> h = pack_host(
      segs, P->Npad, kc, bf16 ? 8 : 4,
      [H, HB](int64_t np) {
        const int ub = (int)(np / (3 * HB)), rem = (int)(np % (3 * HB));
        const int g = rem / HB, j = ub * HB + rem % HB;
        return j < H ? g * H + j : -1;
      },
      &P->Kpad);
  return upload_w(mem, &P->d, h, bf16);
}

// r/z biases summed over both sides; candidate bias split by side.
hipError_t upload_gru_bias(Allocs& mem, GruBias* b, const float* b_in, const float* b_st, int H) {
  std::vector<float> rz(2 * H, 0.f), ni(H, 0.f), ns(H, 0.f);
  for (int j = 0; j < 2 * H; ++j) rz[j] = (b_in ? b_in[j] : 0.f) + (b_st ? b_st[j] : 0.f);
  for (int j = 0; j < H; ++j) {
    ni[j] = b_in ? b_in[2 * H + j] : 0.f;
    ns[j] = b_st ? b_st[2 * H + j] : 0.f;
  }
  hipError_t e = upload(mem, &b->brz, rz.data(), rz.size());
  if (e == hipSuccess) e = upload(mem, &b->bni, ni.data(), ni.size());
  if (e == hipSuccess) e = upload(mem, &b->bns, ns.data(), ns.size());
  return e;
}

// An fp32 activation segment (chunk kc of the model's precision).
ASeg make_seg(const float* p, int64_t ld, int K, int side, int kc) {
  ASeg s{};
  s.p = p;
  s.ld = ld;
  s.K = K;
  s.nchunk = ceil_div(K, kc);
  s.side = side;
  return s;
}

// Embedding rows gathered by id (fp32, or bf16 rows padded to emb_ld).
ASeg emb_seg(const nmt_model* m, const void* table, const int32_t* ids, int nrows) {
  ASeg s{};
  s.p = table;
  s.gather = ids;
  s.gmax = nrows;
  s.ld = m->emb_ld;
  s.K = m->bf16 ? (int)m->emb_ld : m->dims.E;
  s.nchunk = ceil_div(s.K, m->kc);
  s.side = 0;
  s.bf16 = m->bf16 ? 1 : 0;
  return s;
}

AOperand make_a(int M, std::initializer_list<ASeg> segs) {
  AOperand a{};
  a.M = M;
  a.nseg = 0;
  for (const ASeg& s : segs) a.seg[a.nseg++] = s;
  return a;
}

// The model's per-word tables: tab_x = E_tgt . W_x (the first GRU's input
// side, gates [r | z | n]) and tab_y = E_tgt . W_y (the readout's word term),
// one row per target word, computed with the model's GEMM in its precision
// (fp32 sums).  Allocates both tables (kept with the model's other buffers).
hipError_t word_tables(nmt_model* m, hipStream_t st) {
  const nmt_dims& d = m->dims;
  const int V = d.V, E = d.E, H = d.H;
  hipError_t e = m->mem.alloc((void**)&m->tab_x, (size_t)V * 3 * H * 4);
  if (e == hipSuccess) e = m->mem.alloc((void**)&m->tab_y, (size_t)V * E * 4);
  const AOperand A = make_a(V, {emb_seg(m, m->emb_tgt, nullptr, V)});
  if (e == hipSuccess)
    e = launch_gemm_plain(Tile::Large, A, m->g1x, PlainEpi{m->tab_x, 3 * H, nullptr, 3 * H, 0, nullptr, 1}, st);
  if (e == hipSuccess)
    e = launch_gemm_plain(Tile::Large, A, m->roy, PlainEpi{m->tab_y, E, nullptr, E, 0, nullptr, 1}, st);
  return e;
}

nmt_status check_device(const nmt_model* m) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return fail(NMT_EDEVICE, "hipGetDevice failed");
  if (dev != m->device) return fail(NMT_EINVAL, "model lives on device %d but device %d is current", m->device, dev);
  return NMT_OK;
}

nmt_status hip_fail(hipError_t e, const char* what) {
  if (e == hipErrorOutOfMemory) return fail(NMT_ENOMEM, "%s: out of device memory", what);
  return fail(NMT_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

// K split of a small-tile plain GEMM: at least four K chunks per block, and
// enough blocks for about two per CU (measured on the readout at 256 CUs:
// bf16 512 blocks leave B = 4096 unsplit, 6.5 us faster than 2 splits and
// their reduction; fp32 512 rather than 1024 blocks, 2 splits at B = 2000
// and 4 at B = 1000, are 1.5-2 us faster).
int plain_ksplit(int M, int N, int K_total, int kc, Tile t, int cus) {
  const int tiles = ceil_div(M, tile_m(t)) * ceil_div(N, tile_n(t));
  const int nc = ceil_div(K_total, kc);
  int ks = ceil_div(2 * cus, tiles);
  if (ks > nc / 4) ks = nc / 4;
  if (ks > 8) ks = 8;
  return ks < 1 ? 1 : ks;
}

// Workspace layout of one step (offsets in bytes, 256-aligned).  s1 (and
// its bf16 copy) and the context live across the two GRUs; everything from
// q on is dead while a GRU runs, so a GRU's split-K partial sums (gpart)
// reuse that region, extended if they need more.
struct WsLayout {
  size_t s1, s1h, c, q, t, part, kpart, perm, tiles, ntiles, zreq, gpart, total;
  int nS, vtm;        // vocabulary slices and row tile
  int ks_q, ks_ro;    // K splits of the query and readout GEMMs
  int ks_g1, ks_g2;   // K splits of the two GRUs (1: fused cell, no partials)
};

WsLayout ws_layout(const nmt_model* m, int64_t B) {
  const nmt_dims& d = m->dims;
  auto al = [](size_t x) { return (x + 255) / 256 * 256; };
  WsLayout L{};
  size_t off = 0;
  L.s1 = off;
  off += al((size_t)B * d.H * 4);
  // bf16 weights: a bf16 copy of s1 for the GEMMs that read it
  L.s1h = off;
  off += m->bf16 ? al((size_t)B * d.H * 2) : 0;
  L.c = off;  // the context, or (precomp) its products [B x cpw_ld]
  off += al((size_t)B * (m->precomp ? m->cpw_ld : 2 * d.H) * 4);
  L.q = off;
  off += al((size_t)B * d.A * 4);
  L.t = off;
  off += al((size_t)B * d.E * 4);
  L.vtm = vocab_tm((int)B, m->dims.V, m->bf16, m->out.Kpad, m->dims.E, m->out.nbias, m->cus);
  L.nS = vocab_slices((int)B, m->dims.V, m->bf16, m->cus, L.vtm);
  L.part = off;
  off += al((size_t)B * L.nS * sizeof(float2));
  // The query GEMM splits its K where its tiles fit in one round of the CUs
  // (a forest's levels, the phrase loop, B = 1000 at A = 1024), the attention
  // adding the split sums as it loads the query: ruen_b1000 query 27.1 ->
  // 23.1 us, attention +0.4 us (with a reduction kernel of its own, the
  // split had measured slower there, 28 -> 32 us).  At 512 tiles (B = 2000)
  // a split of two measured even.
  const int tiles_q = ceil_div(B, kPlainSmallTM) * ceil_div(d.A, kPlainSmallTN);
  L.ks_q = tiles_q <= m->cus ? plain_ksplit((int)B, d.A, d.H, m->kc, Tile::Small, m->cus) : 1;

  L.ks_ro = plain_ksplit((int)B, d.E, d.H + (m->precomp ? 0 : d.E + 2 * d.H), m->kc, Tile::Small, m->cus);
  size_t kp = 0;
  if (L.ks_q > 1) kp = (size_t)L.ks_q * B * d.A;
  if (L.ks_ro > 1 && (size_t)L.ks_ro * B * d.E > kp) kp = (size_t)L.ks_ro * B * d.E;
  L.kpart = off;
  off += al(kp * 4);
  // attention's grouping of rows by sentence (at most one tile per row)
  L.perm = off;
  off += al((size_t)B * 4);
  L.tiles = off;
  off += al((size_t)B * 16);
  L.ntiles = off;
  off += al(4);
  L.zreq = off;  // the requested words' logits
  off += al((size_t)B * 4);
  // the GRUs' K splits: GRU1 reads [x | s_prev], GRU2 [s1 | c] (precomp:
  // s_prev and s1 alone, their input sides added by the cells)
  const int kc = m->kc;
  const int kx = m->precomp ? 0 : m->bf16 ? (int)m->emb_ld : d.E;
  L.ks_g1 = gru_ksplit((int)B, d.H, ceil_div(kx, kc) + ceil_div(d.H, kc), m->bf16, m->cus);
  L.ks_g2 = gru_ksplit((int)B, d.H, ceil_div(d.H, kc) + (m->precomp ? 0 : ceil_div(2 * d.H, kc)), m->bf16, m->cus);
  const int ks_g = L.ks_g1 > L.ks_g2 ? L.ks_g1 : L.ks_g2;
  L.gpart = L.q;
  if (ks_g > 1) {
    const size_t end = L.gpart + al((size_t)ks_g * B * 4 * d.H * 4);
    off = end > off ? end : off;
  }
  L.total = off;
  return L;
}

// K splits of the encoder's recurrent GRU: its S rows give few tiles
// (S <= 64: 16 column tiles x 2 directions), so each step's K chunks are
// split until the blocks cover the CUs, at least two chunks per split.
int encoder_ksplit(const nmt_model* m, int S) {
  const int base = ceil_div(S, kGruSmallTM) * ceil_div(m->dims.H, gru_hb(m->bf16)) * 2;
  const int nc = ceil_div(m->dims.H, m->kc);
  int ks = m->cus / base;
  if (ks > nc / 2) ks = nc / 2;
  return ks < 1 ? 1 : ks;
}

nmt_status new_source(nmt_model* m, int32_t S, int32_t Tpad, const int32_t* h_len, bool with_scratch,
                      hipStream_t st, nmt_source** out) {
  const nmt_dims& d = m->dims;
  if (S < 1) return fail(NMT_EINVAL, "S must be >= 1 (got %d)", S);
  if (Tpad < 1 || Tpad > kMaxTpad) return fail(NMT_EINVAL, "Tpad must be in [1, %d] (got %d)", kMaxTpad, Tpad);
  if (!h_len) return fail(NMT_EINVAL, "h_len is NULL");
  for (int s = 0; s < S; ++s)
    if (h_len[s] < 1 || h_len[s] > Tpad)
      return fail(NMT_EINVAL, "h_len[%d] = %d is outside [1, Tpad = %d]", s, h_len[s], Tpad);
  nmt_source* src = new nmt_source();
  src->S = S;
  src->Tpad = Tpad;
  src->H = d.H;
  src->A = d.A;
  src->cpw_ld = m->precomp ? m->cpw_ld : 0;
  src->h_len.assign(h_len, h_len + S);
  const size_t rows = (size_t)S * Tpad;
  hipError_t e = src->mem.alloc((void**)&src->ctx, rows * 2 * d.H * sizeof(float));
  if (e == hipSuccess) e = src->mem.alloc((void**)&src->pctx, rows * d.A * sizeof(float));
  if (e == hipSuccess) e = src->mem.alloc((void**)&src->kfac, rows * d.A * sizeof(float));
  if (e == hipSuccess && m->precomp) e = src->mem.alloc((void**)&src->cproj, rows * m->cpw_ld * sizeof(float));
  if (e == hipSuccess) e = src->mem.alloc((void**)&src->len, S * sizeof(int32_t));
  if (e == hipSuccess) e = src->mem.alloc((void**)&src->kbig, S * sizeof(int32_t));
  if (e == hipSuccess && with_scratch) e = src->mem.alloc((void**)&src->scratch, rows * 6 * d.H * sizeof(float));
  if (e == hipSuccess && with_scratch) {
    src->enc_ks = encoder_ksplit(m, S);
    if (src->enc_ks > 1)
      e = src->mem.alloc((void**)&src->gru_part, (size_t)2 * src->enc_ks * S * 4 * d.H * sizeof(float));
  }
  if (e == hipSuccess)
    e = hipMemcpyAsync(src->len, src->h_len.data(), S * sizeof(int32_t), hipMemcpyHostToDevice, st);
  if (e != hipSuccess) {
    src->mem.release();
    delete src;
    return hip_fail(e, "source allocation");
  }
  *out = src;
  return NMT_OK;
}

// Attention keys pctx = ctx att_Wc + att_b for the unmasked positions, and
// their factors 2^{2 log2(e) pctx} that the score kernels use.
hipError_t source_keys(nmt_model* m, nmt_source* src, hipStream_t st) {
  const nmt_dims& d = m->dims;
  const int C = 2 * d.H;
  AOperand A = make_a(src->S * src->Tpad, {make_seg(src->ctx, C, C, 0, m->kc)});
  PlainEpi ep{src->pctx, d.A, m->att_b, d.A, 0, src->len, src->Tpad};
  hipError_t e = launch_gemm_plain(Tile::Large, A, m->att_Wc, ep, st);
  if (e == hipSuccess) e = launch_key_factors(src->S, src->Tpad, d.A, src->pctx, src->kfac, src->kbig, st);
  if (e == hipSuccess && m->precomp) {
    // the context's products, projected per position (zeros past the length)
    PlainEpi pe{src->cproj, m->cpw_ld, nullptr, m->cpw_ld, 0, src->len, src->Tpad};
    e = launch_gemm_plain(Tile::Large, A, m->cpw, pe, st);
  }
  return e;
}

// Scratch of nmt_score_batch_noalloc: a file-scope device array, so that
// step allocates nothing.  Every GPU the library runs on holds its own copy
// until the process ends.  In host code `scratch` names a host-side stand-in,
// never the device memory: the device address of each GPU's copy is looked
// up once per device (noalloc_scratch, called from nmt_model_create with the
// model's device current) and only that address reaches the kernels.
static __device__ __align__(256) char scratch[NMT_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

hipError_t noalloc_scratch(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || ((uintptr_t)p & 255)) return hipErrorInvalidSymbol;
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return hipSuccess;
}

}  // namespace

namespace nmt {

hipError_t device_malloc(void** p, size_t bytes) {
  int64_t b = g_alloc_budget.load();
  while (b >= 0) {
    if (b == 0) {
      *p = nullptr;
      return hipErrorOutOfMemory;
    }
    if (g_alloc_budget.compare_exchange_weak(b, b - 1)) break;
  }
  const hipError_t e = hipMalloc(p, bytes);
  if (e == hipSuccess) ++g_live_allocs;
  return e;
}

void device_free(void* p) {
  if (!p) return;
  if (hipFree(p) == hipSuccess) --g_live_allocs;
}

}  // namespace nmt

extern "C" {

int64_t nmt_debug_alloc_hook(int32_t fail_after) {
  g_alloc_budget.store(fail_after < 0 ? -1 : fail_after);
  return g_live_allocs.load();
}

int32_t nmt_debug_gemm_form(int32_t form) {
  if (form < 0 || form > 4) return -1;
  return nmt::g_gemm_form.exchange(form);
}

int64_t nmt_debug_gemm_streamed(void) { return nmt::g_gemm_streamed.load(); }

int32_t nmt_debug_precompute(int32_t on) {
  if (on != 0 && on != 1) return -1;
  return g_precompute.exchange(on);
}

const char* nmt_last_error(void) { return g_err.c_str(); }

nmt_status nmt_model_create(const nmt_dims* dims, const nmt_weights* w, nmt_model** out) {
  if (!dims || !w || !out) return fail(NMT_EINVAL, "NULL argument");
  *out = nullptr;
  const nmt_dims d = *dims;
  if (d.V_src <= 0 || d.V <= 0 || d.E <= 0 || d.H <= 0 || d.A <= 0)
    return fail(NMT_EINVAL, "dimensions must be positive");
  if (d.E % 4 || d.H % 4 || d.A % 4) return fail(NMT_EINVAL, "E, H and A must be multiples of 4");
  if (d.A > 8 * 256) return fail(NMT_EINVAL, "A must be at most 2048");
  if (d.wtype != NMT_F32 && d.wtype != NMT_BF16) return fail(NMT_EINVAL, "unknown weight type %d", d.wtype);
  const bool bf16 = d.wtype == NMT_BF16;
  if (round_up(d.E + vocab_bias_rows(bf16), chunk_k(bf16)) > vocab_max_kpad(bf16))
    return fail(NMT_EINVAL, "E must be at most %d for this weight type",
                vocab_max_kpad(bf16) - vocab_bias_rows(bf16));
  if (!vocab_offsets_fit(round_up(d.E + vocab_bias_rows(bf16), chunk_k(bf16)), round_up(d.V, kVocabTN) + kVocabSpare,
                         bf16))
    return fail(NMT_EINVAL, "the packed output weights (E x V) must stay under 2 GiB");
  const float* const* wp = (const float* const*)w;
  for (size_t i = 0; i < sizeof(nmt_weights) / sizeof(float*); ++i)
    if (!wp[i]) return fail(NMT_EINVAL, "weight #%zu is NULL", i);

  nmt_model* m = new nmt_model();
  m->dims = d;
  if (hipGetDevice(&m->device) != hipSuccess) {
    delete m;
    return fail(NMT_EDEVICE, "hipGetDevice failed");
  }
  if (hipDeviceGetAttribute(&m->cus, hipDeviceAttributeMultiprocessorCount, m->device) != hipSuccess ||
      m->cus < 1) {
    delete m;
    return fail(NMT_EDEVICE, "cannot read the compute-unit count of device %d", m->device);
  }
  const int E = d.E, H = d.H, A = d.A, C = 2 * d.H, V = d.V;
  hipError_t e = hipSuccess;
  auto step = [&](hipError_t r) {
    if (e == hipSuccess) e = r;
  };
  m->bf16 = bf16;
  m->kc = chunk_k(bf16);
  m->emb_ld = bf16 ? round_up(E, PrecBF16::KV) : E;
  const int kc = m->kc;
  step(upload_table(m->mem, &m->emb_src, w->emb_src, d.V_src, E, m->emb_ld, bf16));
  step(upload_table(m->mem, &m->emb_tgt, w->emb_tgt, V, E, m->emb_ld, bf16));
  {  // encoder input projections of both directions side by side: [E x 6H]
    std::vector<float> Win((size_t)E * 6 * H), bin((size_t)6 * H);
    for (int k = 0; k < E; ++k)
      for (int j = 0; j < 3 * H; ++j) {
        Win[(size_t)k * 6 * H + j] = w->enc_f_W[(size_t)k * 3 * H + j];
        Win[(size_t)k * 6 * H + 3 * H + j] = w->enc_b_W[(size_t)k * 3 * H + j];
      }
    for (int j = 0; j < 3 * H; ++j) {
      bin[j] = w->enc_f_b[j];
      bin[3 * H + j] = w->enc_b_b[j];
    }
    if (e == hipSuccess) step(pack_plain(m->mem, &m->enc_in, {{Win.data(), E, 6 * H}}, 6 * H, kPlainLargeTN, kc, bf16));
    step(upload(m->mem, &m->enc_in_b, bin.data(), bin.size()));
  }
  if (e == hipSuccess) step(pack_gru(m->mem, &m->enc_U[0], {{w->enc_f_U, H, 3 * H}}, H, kc, bf16));
  if (e == hipSuccess) step(pack_gru(m->mem, &m->enc_U[1], {{w->enc_b_U, H, 3 * H}}, H, kc, bf16));
  if (e == hipSuccess) step(upload_gru_bias(m->mem, &m->enc_bias, nullptr, nullptr, H));
  if (e == hipSuccess) step(pack_plain(m->mem, &m->att_Wc, {{w->att_Wc, C, A}}, A, kPlainLargeTN, kc, bf16));
  step(upload(m->mem, &m->att_b, w->att_b, A));
  if (e == hipSuccess) step(pack_plain(m->mem, &m->init_W, {{w->init_W, C, H}}, H, kPlainSmallTN, kc, bf16));
  step(upload(m->mem, &m->init_b, w->init_b, H));
  m->precomp = !bf16 && g_precompute.load() != 0;
  if (m->precomp) {
    if (e == hipSuccess) step(pack_gru(m->mem, &m->g1, {{w->g1_U, H, 3 * H}}, H, kc, bf16));
    if (e == hipSuccess) step(pack_plain(m->mem, &m->g1x, {{w->g1_W, E, 3 * H}}, 3 * H, kPlainLargeTN, kc, bf16));
  } else if (e == hipSuccess) {
    step(pack_gru(m->mem, &m->g1, {{w->g1_W, E, 3 * H}, {w->g1_U, H, 3 * H}}, H, kc, bf16));
  }
  if (e == hipSuccess) step(upload_gru_bias(m->mem, &m->g1_bias, w->g1_b, nullptr, H));
  if (e == hipSuccess) step(pack_plain(m->mem, &m->att_Wq, {{w->att_Wq, H, A}}, A, kPlainSmallTN, kc, bf16));
  step(upload(m->mem, &m->att_v, w->att_v, A));
  if (m->precomp) {
    if (e == hipSuccess) step(pack_gru(m->mem, &m->g2, {{w->g2_U, H, 3 * H}}, H, kc, bf16));
    // [g2_Wc | ro_Wc]: C x (3H + E)
    std::vector<float> cw((size_t)C * (3 * H + E));
    for (int k = 0; k < C; ++k) {
      memcpy(&cw[(size_t)k * (3 * H + E)], w->g2_Wc + (size_t)k * 3 * H, sizeof(float) * 3 * H);
      memcpy(&cw[(size_t)k * (3 * H + E) + 3 * H], w->ro_Wc + (size_t)k * E, sizeof(float) * E);
    }
    if (e == hipSuccess) step(pack_plain(m->mem, &m->cpw, {{cw.data(), C, 3 * H + E}}, 3 * H + E, kPlainLargeTN, kc, bf16));
    m->cpw_ld = (int)m->cpw.Npad;
  } else if (e == hipSuccess) {
    step(pack_gru(m->mem, &m->g2, {{w->g2_U, H, 3 * H}, {w->g2_Wc, C, 3 * H}}, H, kc, bf16));
  }
  if (e == hipSuccess) step(upload_gru_bias(m->mem, &m->g2_bias, nullptr, w->g2_b, H));
  if (m->precomp) {
    if (e == hipSuccess) step(pack_plain(m->mem, &m->ro, {{w->ro_Ws, H, E}}, E, kPlainSmallTN, kc, bf16));
    if (e == hipSuccess) step(pack_plain(m->mem, &m->roy, {{w->ro_Wy, E, E}}, E, kPlainLargeTN, kc, bf16));
  } else if (e == hipSuccess) {
    step(pack_plain(m->mem, &m->ro, {{w->ro_Ws, H, E}, {w->ro_Wy, E, E}, {w->ro_Wc, C, E}}, E, kPlainSmallTN, kc, bf16));
  }
  step(upload(m->mem, &m->ro_b, w->ro_b, E));
  if (e == hipSuccess) {
    // output weights with the bias as extra rows (see vocab_bias_rows)
    const int nb = vocab_bias_rows(bf16);
    std::vector<float> brows((size_t)nb * V);
    for (int v = 0; v < V; ++v) {
      const float b = w->out_b[v];
      if (!bf16) {
        brows[(size_t)v] = b;
      } else {
        const float hi = bf16_value(b), mid = bf16_value(b - hi);
        brows[(size_t)v] = hi;
        brows[(size_t)V + v] = mid;
        brows[(size_t)2 * V + v] = b - hi - mid;  // exact in bf16: what remains has at most 8 significant bits
      }
    }
    Seg sg{w->out_W, E, V, brows.data(), nb};
    step(pack_plain(m->mem, &m->out, {sg}, V, kVocabTN, kc, bf16, kVocabSpare));
    m->out.Krows = E;
    m->out.nbias = nb;
  }
  if (e == hipSuccess && m->precomp) step(word_tables(m, nullptr));
  step(m->mem.alloc((void**)&m->err, sizeof(int)));
  if (e == hipSuccess) step(hipMemset(m->err, 0, sizeof(int)));
  if (e == hipSuccess) step(noalloc_scratch(m->device, &m->noalloc_ws));
  if (e == hipSuccess) step(hipDeviceSynchronize());
  if (e != hipSuccess) {
    m->mem.release();
    delete m;
    return hip_fail(e, "nmt_model_create");
  }
  *out = m;
  return ok();
}

static void drop_profile_events(nmt_model* m) {
  for (hipEvent_t ev : m->prof_events) (void)hipEventDestroy(ev);
  m->prof_events.clear();
  m->prof_on = false;
  m->prof_max = m->prof_used = 0;
}

void nmt_model_destroy(nmt_model* m) {
  if (!m) return;
  (void)hipDeviceSynchronize();
  drop_profile_events(m);
  m->mem.release();
  delete m;
}

nmt_status nmt_encode(nmt_model* m, int32_t S, int32_t Tpad, const int32_t* d_src_ids, const int32_t* h_len,
                      float* d_s0_out, void* stream, nmt_source** out) {
  if (!m || !out) return fail(NMT_EINVAL, "NULL model or output");
  *out = nullptr;
  if (!d_src_ids) return fail(NMT_EINVAL, "d_src_ids is NULL");
  if (d_s0_out && !aligned16(d_s0_out)) return fail(NMT_EINVAL, "d_s0_out must be 16-byte aligned");
  nmt_status rc = check_device(m);
  if (rc != NMT_OK) return rc;
  hipStream_t st = (hipStream_t)stream;
  nmt_source* src = nullptr;
  rc = new_source(m, S, Tpad, h_len, true, st, &src);
  if (rc != NMT_OK) return rc;
  const nmt_dims& d = m->dims;
  const int E = d.E, H = d.H, C = 2 * H;
  const int64_t rows = (int64_t)S * Tpad;
  float* Xp = src->scratch;  // [S*Tpad x 6H] input-side pre-activations of both directions
  hipError_t e = launch_check_src_ids(S, Tpad, d_src_ids, src->len, d.V_src, m->err, st);
  if (e == hipSuccess) {
    AOperand A = make_a((int)rows, {emb_seg(m, m->emb_src, d_src_ids, d.V_src)});
    PlainEpi ep{Xp, 6 * H, m->enc_in_b, 6 * H, 0, nullptr, 1};
    e = launch_gemm_plain(Tile::Large, A, m->enc_in, ep, st);
  }
  // The recurrence: step t runs the forward direction at position t and the
  // backward direction at position Tpad-1-t in one launch.  Positions at or
  // past a sentence's length are written as zeros, which is also the
  // backward direction's initial state there.
  const int64_t ldc = (int64_t)Tpad * C, ldx = (int64_t)Tpad * 6 * H;
  for (int t = 0; t < Tpad && e == hipSuccess; ++t) {
    GruProblem p[2];
    for (int dir = 0; dir < 2; ++dir) {
      const int pos = dir == 0 ? t : Tpad - 1 - t;
      const int prev = dir == 0 ? pos - 1 : pos + 1;
      const bool has_prev = prev >= 0 && prev < Tpad;
      const float* hprev = has_prev ? src->ctx + (int64_t)prev * C + dir * H : nullptr;
      GruProblem& g = p[dir];
      g.A = has_prev ? make_a(S, {make_seg(hprev, ldc, H, 1, m->kc)}) : make_a(S, {});
      g.Wp = m->enc_U[dir].d;
      g.Npad = m->enc_U[dir].Npad;
      g.ep = GruEpi{hprev, ldc, nullptr, 0, Xp + (int64_t)pos * 6 * H + dir * 3 * H, ldx, m->enc_bias.brz, m->enc_bias.bni,
                    m->enc_bias.bns, src->ctx + (int64_t)pos * C + dir * H, ldc, src->len, pos, H};
    }
    const bool split = src->enc_ks > 1 && p[0].A.nseg > 0 && p[1].A.nseg > 0;
    e = split ? launch_gemm_gru_split(p, 2, H, m->bf16, src->enc_ks, src->gru_part, S, kGruSmallTM, st)
              : launch_gemm_gru(p, 2, H, m->bf16, m->cus, st);
  }
  if (e == hipSuccess) e = source_keys(m, src, st);
  if (e == hipSuccess && d_s0_out) {
    float* mean = Xp;  // the pre-activations are consumed by now (stream order)
    e = launch_masked_mean(S, Tpad, C, src->ctx, src->len, mean, st);
    if (e == hipSuccess) {
      AOperand A = make_a(S, {make_seg(mean, C, C, 0, m->kc)});
      PlainEpi ep{d_s0_out, H, m->init_b, H, 1, nullptr, 1};
      e = launch_gemm_plain(Tile::Small, A, m->init_W, ep, st);
    }
  }
  if (e != hipSuccess) {
    (void)hipStreamSynchronize(st);
    nmt_source_destroy(src);
    return hip_fail(e, "nmt_encode");
  }
  *out = src;
  return ok();
}

nmt_status nmt_source_from_annotations(nmt_model* m, int32_t S, int32_t Tpad, const float* d_ctx,
                                       const int32_t* h_len, void* stream, nmt_source** out) {
  if (!m || !out) return fail(NMT_EINVAL, "NULL model or output");
  *out = nullptr;
  if (!d_ctx || !aligned16(d_ctx)) return fail(NMT_EINVAL, "d_ctx must be a 16-byte aligned device pointer");
  nmt_status rc = check_device(m);
  if (rc != NMT_OK) return rc;
  hipStream_t st = (hipStream_t)stream;
  nmt_source* src = nullptr;
  rc = new_source(m, S, Tpad, h_len, false, st, &src);
  if (rc != NMT_OK) return rc;
  hipError_t e = launch_masked_copy(S, Tpad, 2 * m->dims.H, d_ctx, src->len, src->ctx, st);
  if (e == hipSuccess) e = source_keys(m, src, st);
  if (e != hipSuccess) {
    (void)hipStreamSynchronize(st);
    nmt_source_destroy(src);
    return hip_fail(e, "nmt_source_from_annotations");
  }
  *out = src;
  return ok();
}

nmt_status nmt_source_info(const nmt_source* src, int32_t* S, int32_t* Tpad, const float** d_ctx,
                           const float** d_pctx) {
  if (!src) return fail(NMT_EINVAL, "NULL source");
  if (S) *S = src->S;
  if (Tpad) *Tpad = src->Tpad;
  if (d_ctx) *d_ctx = src->ctx;
  if (d_pctx) *d_pctx = src->pctx;
  return ok();
}

void nmt_source_destroy(nmt_source* src) {
  if (!src) return;
  (void)hipDeviceSynchronize();
  src->mem.release();
  delete src;
}

size_t nmt_score_workspace_bytes(const nmt_model* m, int32_t B) {
  if (!m || B <= 0) return 0;
  // Some smaller batches need more bytes than B itself: the vocabulary
  // kernel may take more slices for them (more partials per row), the
  // readout more K splits.  Both choices are fixed within a run of batch
  // sizes that fill the same number of row tiles (tiles of 64 or 128 rows,
  // multiples of 32), where the largest size needs the most.  So the
  // maximum over B and every multiple of 32 below it bounds every smaller
  // call, and a workspace sized for B serves any batch up to B (a forest's
  // levels, a shrinking batch).
  size_t mx = ws_layout(m, B).total;
  for (int32_t b = 32; b < B; b += 32) {
    const size_t t = ws_layout(m, b).total;
    if (t > mx) mx = t;
  }
  return mx;
}

}  // extern "C"

namespace {

// One batched decoder step (the forward step of Section 5.1) for B rows.
// Row b's input state is row state_row[b] of the state pool (row b when
// state_row is NULL), its previous word y_prev[b], and its requested words
// are given by rq.  Debug outputs are optional.
nmt_status score_step(nmt_model* m, const nmt_source* src, int32_t B, const float* pool, int32_t pool_rows,
                      const int32_t* state_row, const int32_t* d_y_prev, const int32_t* d_sent_id, Requests rq,
                      float* d_logp, float* d_s_new, float* d_logZ, void* d_workspace, size_t ws_bytes, hipStream_t st,
                      float* d_alpha, float* d_c, float* d_s1, float* d_t, const AttnGroups* pre_grp = nullptr) {
  const WsLayout L = ws_layout(m, B);
  if (!d_workspace || ((uintptr_t)d_workspace & 255)) return fail(NMT_EINVAL, "workspace must be 256-byte aligned");
  if (ws_bytes < L.total) return fail(NMT_EWORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, L.total);
  // the source's arrays have the widths of the model that set it up, and
  // hold the annotations' projections only for a model that mixes them
  if (src->H != m->dims.H || src->A != m->dims.A)
    return fail(NMT_EINVAL, "the source was set up for a model with H = %d, A = %d (this one: %d, %d)", src->H,
                src->A, m->dims.H, m->dims.A);
  if (m->precomp != (src->cproj != nullptr) || src->cpw_ld != (m->precomp ? m->cpw_ld : 0))
    return fail(NMT_EINVAL, "the source was set up for a model %s the annotations' projections",
                src->cproj ? "with" : "without");
  nmt_status rc = check_device(m);
  if (rc != NMT_OK) return rc;

  const nmt_dims& d = m->dims;
  const int E = d.E, H = d.H, Aw = d.A, C = 2 * H, V = d.V;
  char* ws = (char*)d_workspace;
  float* s1 = (float*)(ws + L.s1);
  float* q = (float*)(ws + L.q);
  float* c = (float*)(ws + L.c);
  // With bf16 weights the context is kept in bf16: the two GEMMs that read
  // it round it to bf16 anyway, so the values are the same, and its stores
  // and the GEMMs' loads of it move half the bytes (bf16_b4096: GRU2 114 ->
  // 107 us, readout 56 -> 49 us, attention 78 -> 74 us).
  const bool c16 = m->bf16;
  ASeg c_seg = make_seg(c, C, C, 0, m->kc);
  c_seg.bf16 = c16 ? 1 : 0;
  // GRU1 also writes s1 in bf16 for the query and GRU2's state operand (the
  // cell of GRU2 reads the fp32 s1): query 34 -> 27 us, GRU2 107 -> 105 us,
  // GRU1 +1 us for the extra stores.  Its rows are H wide, not padded: a
  // vector that runs past H reads the next row's (finite) values against
  // zero weights.  A bf16 copy of the new state for the readout gained less
  // than its stores cost in GRU2.
  __bf16* s1h = m->bf16 ? (__bf16*)(ws + L.s1h) : nullptr;
  auto state_seg = [&](const float* f32, const __bf16* b16, int side) {
    ASeg sg = make_seg(b16 ? (const float*)b16 : f32, H, H, side, m->kc);
    sg.bf16 = b16 ? 1 : 0;
    return sg;
  };
  float* t = (float*)(ws + L.t);
  float2* part = (float2*)(ws + L.part);
  ASeg h_seg = make_seg(pool, H, H, 1, m->kc);             // H_{i-1}: input states, gathered by row
  h_seg.gather = state_row;
  h_seg.gmax = pool_rows;
  hipEvent_t* ev = nullptr;
  if (m->prof_on && m->prof_used < m->prof_max) ev = &m->prof_events[(size_t)(m->prof_used++) * (NMT_NUM_PHASES + 1)];
  hipError_t e = hipSuccess;
  auto mark = [&](int i) {
    if (ev && e == hipSuccess) e = hipEventRecord(ev[i], st);
  };
  mark(0);

  // first GRU: s1 = GRU(x, s_prev), x = E_i the embeddings of the previous
  // words (ids outside the vocabulary, and -1, read zeros), or with the
  // model's tables their products with the input-side weights, rows y_prev
  // of the table
  const ASeg x_seg = emb_seg(m, m->emb_tgt, d_y_prev, V);
  GruProblem g1;
  g1.A = m->precomp ? make_a(B, {h_seg}) : make_a(B, {x_seg, h_seg});
  g1.Wp = m->g1.d;
  g1.Npad = m->g1.Npad;
  g1.ep = GruEpi{pool, H, state_row, pool_rows, nullptr, 0, m->g1_bias.brz, m->g1_bias.bni, m->g1_bias.bns,
                 s1, H, nullptr, 0, H};
  g1.ep.out16 = s1h;
  if (m->precomp) {
    g1.ep.xin = m->tab_x;
    g1.ep.ldx = 3 * H;
    g1.ep.xrow = d_y_prev;
    g1.ep.xrows = V;
  }
  float* gpart = (float*)(ws + L.gpart);
  auto run_gru = [&](const GruProblem& g, int ks) {
    // (the test switch's forced streaming skips the K split, which the
    // streamed form never takes, so that small batches reach it)
    return ks > 1 && !gemm_stream_forced(g_gemm_form.load(std::memory_order_relaxed))
               ? launch_gemm_gru_split(&g, 1, H, m->bf16, ks, gpart, B, gru_split_tm(B, H, m->bf16, m->cus), st)
                  : launch_gemm_gru(&g, 1, H, m->bf16, m->cus, st);
  };
  if (e == hipSuccess) e = run_gru(g1, L.ks_g1);
  mark(NMT_PHASE_GRU1 + 1);
  // attention query q = s1 att_Wq
  QuerySrc qsrc{q, 1, 0};
  if (e == hipSuccess) {
    PlainEpi ep{q, Aw, nullptr, Aw, 0, nullptr, 1, L.ks_q, (float*)(ws + L.kpart)};
    // a split query leaves its sums for the attention to add as it loads
    // them (the test switch's forced streaming writes q itself)
    ep.defer_reduce = L.ks_q > 1 && !gemm_stream_forced(g_gemm_form.load(std::memory_order_relaxed));
    e = launch_gemm_plain(Tile::Small, make_a(B, {state_seg(s1, s1h, 0)}), m->att_Wq, ep, st, m->cus);
    qsrc = ep.defer_reduce ? QuerySrc{ep.part, L.ks_q, (int64_t)B * Aw} : QuerySrc{q, 1, 0};
  }
  mark(NMT_PHASE_QUERY + 1);
  // masked attention and context
  if (e == hipSuccess) {
    // (a forest's levels come with their grouping done, all in one launch)
    const AttnGroups grp =
        pre_grp ? *pre_grp : AttnGroups{(int32_t*)(ws + L.perm), (int4*)(ws + L.tiles), (int32_t*)(ws + L.ntiles)};
    auto attend = [&](const float* X, int width, float* out, float* alpha_out, bool out16) {
      return launch_attention(B, Aw, width, src->Tpad, qsrc, src->kfac, src->pctx, src->kbig, X, src->len, d_sent_id,
                              src->S, m->att_v, out, alpha_out, grp, out16, m->cus, st, pre_grp != nullptr);
    };
    // precomp: the attention mixes the annotations' projections, giving the
    // context's products with the second GRU's and the readout's weights;
    // the context itself only for the debug output (the same weights over
    // the annotations, while the query is still in place)
    if (m->precomp) {
      e = attend(src->cproj, m->cpw_ld, c, d_alpha, false);
      if (e == hipSuccess && d_c) e = attend(src->ctx, C, d_c, nullptr, false);
    } else {
      e = attend(src->ctx, C, c, d_alpha, c16);
    }
  }
  mark(NMT_PHASE_ATTENTION + 1);
  // second GRU: s_new = GRU(c, s1) (precomp: its input side c W_c from the attention)
  if (e == hipSuccess) {
    GruProblem g2;
    g2.A = m->precomp ? make_a(B, {state_seg(s1, s1h, 1)}) : make_a(B, {state_seg(s1, s1h, 1), c_seg});
    g2.Wp = m->g2.d;
    g2.Npad = m->g2.Npad;
    g2.ep = GruEpi{s1, H, nullptr, 0, nullptr, 0, m->g2_bias.brz, m->g2_bias.bni, m->g2_bias.bns, d_s_new, H,
                   nullptr, 0, H};
    if (m->precomp) {
      g2.ep.xin = c;
      g2.ep.ldx = m->cpw_ld;
    }
    e = run_gru(g2, L.ks_g2);
  }
  mark(NMT_PHASE_GRU2 + 1);
  // readout t = tanh(s_new Ws + x Wy + c Wc + b), with the model's tables
  // the word term x Wy from a table like the first GRU's input side
  if (e == hipSuccess) {
    PlainEpi ep{t, E, m->ro_b, E, 1, nullptr, 1, L.ks_ro, (float*)(ws + L.kpart)};
    if (m->precomp) {  // the word term from its table, the context term from the attention
      ep.add = m->tab_y;
      ep.ld_add = E;
      ep.add_row = d_y_prev;
      ep.add_rows = V;
      ep.add2 = c + 3 * H;
      ep.ld_add2 = m->cpw_ld;
    }
    if (m->bf16) {  // the vocabulary and combine kernels stage t in bf16 anyway
      ep.out16 = (__bf16*)t;
      ep.ldo = bf16_row(E);
    }
    e = launch_gemm_plain(Tile::Small,
                          m->precomp ? make_a(B, {make_seg(d_s_new, H, H, 0, m->kc)})
                                     : make_a(B, {make_seg(d_s_new, H, H, 0, m->kc), x_seg, c_seg}),
                          m->ro,
                          ep, st, m->cus);
  }
  mark(NMT_PHASE_READOUT + 1);
  // vocabulary projection with an online log-sum-exp per slice, then the combine
  // rows with one request: the vocabulary kernel also picks out its logit
  float* zreq = rq.req ? (float*)(ws + L.zreq) : nullptr;
  if (e == hipSuccess)
    e = launch_vocab_lse(t, m->bf16, B, E, m->out, V, part, L.nS, L.vtm, rq.req, rq.req_off, rq.nreq, zreq, st);
  mark(NMT_PHASE_VOCAB + 1);
  if (e == hipSuccess)
    e = launch_lse_combine(B, part, L.nS, t, m->bf16, E, m->out, V, rq, d_y_prev, d_sent_id, src->S, d_logp, d_logZ,
                           m->err, zreq, st);
  mark(NMT_PHASE_COMBINE + 1);
  if (e == hipSuccess && d_s1) e = hipMemcpyAsync(d_s1, s1, (size_t)B * H * 4, hipMemcpyDeviceToDevice, st);
  if (e == hipSuccess && d_c && !m->precomp)
    e = c16 ? launch_bf16_to_f32(c, B, C, C, d_c, st)
            : hipMemcpyAsync(d_c, c, (size_t)B * C * 4, hipMemcpyDeviceToDevice, st);
  if (e == hipSuccess && d_t)
    e = m->bf16 ? launch_bf16_to_f32(t, B, E, bf16_row(E), d_t, st)
                : hipMemcpyAsync(d_t, t, (size_t)B * E * 4, hipMemcpyDeviceToDevice, st);
  if (e != hipSuccess) return hip_fail(e, "score step");
  return ok();
}

}  // namespace

extern "C" {

nmt_status nmt_score_batch_debug(nmt_model* m, const nmt_source* src, int32_t B, const float* d_s_prev,
                                 const int32_t* d_y_prev, const int32_t* d_sent_id, const int32_t* d_req,
                                 float* d_logp, float* d_s_new, float* d_logZ, void* d_workspace, size_t ws_bytes,
                                 void* stream, float* d_alpha, float* d_c, float* d_s1, float* d_t) {
  if (!m || !src) return fail(NMT_EINVAL, "NULL model or source");
  if (B < 0) return fail(NMT_EINVAL, "B must be >= 0 (got %d)", B);
  if (B == 0) return ok();
  if (!d_s_prev || !d_y_prev || !d_sent_id || !d_req || !d_logp || !d_s_new)
    return fail(NMT_EINVAL, "a required device pointer is NULL");
  if (!aligned16(d_s_prev) || !aligned16(d_s_new))
    return fail(NMT_EINVAL, "d_s_prev and d_s_new must be 16-byte aligned");
  if ((d_c && !aligned16(d_c)) || (d_s1 && !aligned16(d_s1)) || (d_t && !aligned16(d_t)))
    return fail(NMT_EINVAL, "debug outputs must be 16-byte aligned");
  Requests rq{nullptr, d_req, B, nullptr, 0};
  return score_step(m, src, B, d_s_prev, B, nullptr, d_y_prev, d_sent_id, rq, d_logp, d_s_new, d_logZ, d_workspace,
                    ws_bytes, (hipStream_t)stream, d_alpha, d_c, d_s1, d_t);
}

nmt_status nmt_score_batch(nmt_model* m, const nmt_source* src, int32_t B, const float* d_s_prev,
                           const int32_t* d_y_prev, const int32_t* d_sent_id, const int32_t* d_req, float* d_logp,
                           float* d_s_new, float* d_logZ, void* d_workspace, size_t ws_bytes, void* stream) {
  return nmt_score_batch_debug(m, src, B, d_s_prev, d_y_prev, d_sent_id, d_req, d_logp, d_s_new, d_logZ, d_workspace,
                               ws_bytes, stream, nullptr, nullptr, nullptr, nullptr);
}

nmt_status nmt_score_batch_noalloc(nmt_model* m, const nmt_source* src, int32_t B, const float* d_s_prev,
                                   const int32_t* d_y_prev, const int32_t* d_sent_id, const int32_t* d_req,
                                   float* d_logp, float* d_s_new, float* d_logZ, void* stream) {
  if (!m || !src) return fail(NMT_EINVAL, "NULL model or source");
  if (B < 0) return fail(NMT_EINVAL, "B must be >= 0 (got %d)", B);
  if (B == 0) return ok();
  if (!m->noalloc_ws) return fail(NMT_EDEVICE, "the allocation-free scratch of device %d is not set up", m->device);
  const size_t need = ws_layout(m, B).total;
  if (need > (size_t)NMT_NOALLOC_SCRATCH_BYTES)
    return fail(NMT_EWORKSPACE, "%d rows need %zu bytes of scratch; the allocation-free step holds %zu (use "
                "nmt_score_batch with a workspace, or fewer rows)", B, need, (size_t)NMT_NOALLOC_SCRATCH_BYTES);
  return nmt_score_batch(m, src, B, d_s_prev, d_y_prev, d_sent_id, d_req, d_logp, d_s_new, d_logZ, m->noalloc_ws,
                         (size_t)NMT_NOALLOC_SCRATCH_BYTES, stream);
}

nmt_status nmt_score_forest_step(nmt_model* m, const nmt_source* src, int32_t B, const float* d_state_pool,
                                 int32_t pool_rows, const int32_t* d_state_row, const int32_t* d_y_prev,
                                 const int32_t* d_sent_id, const int32_t* d_req_off, const int32_t* d_req,
                                 int32_t nreq, float* d_logp, float* d_s_new, float* d_logZ, void* d_workspace,
                                 size_t ws_bytes, void* stream) {
  if (!m || !src) return fail(NMT_EINVAL, "NULL model or source");
  if (B < 0 || nreq < 0 || pool_rows < 0) return fail(NMT_EINVAL, "negative size");
  if (B == 0) return ok();
  if (!d_state_pool || !d_state_row || !d_y_prev || !d_sent_id || !d_req_off || (nreq > 0 && (!d_req || !d_logp)) ||
      !d_s_new)
    return fail(NMT_EINVAL, "a required device pointer is NULL");
  if (!aligned16(d_state_pool) || !aligned16(d_s_new))
    return fail(NMT_EINVAL, "d_state_pool and d_s_new must be 16-byte aligned");
  Requests rq{d_req_off, d_req, nreq, d_state_row, pool_rows};
  return score_step(m, src, B, d_state_pool, pool_rows, d_state_row, d_y_prev, d_sent_id, rq, d_logp, d_s_new, d_logZ,
                    d_workspace, ws_bytes, (hipStream_t)stream, nullptr, nullptr, nullptr, nullptr);
}

// ------------------------------------------------------ several models

// Every device pointer field of a model that refers to a parameter buffer.
static std::vector<void**> param_fields(nmt_model* m) {
  std::vector<void**> f = {&m->emb_src, &m->emb_tgt};
  for (Packed* P : {&m->enc_in, &m->enc_U[0], &m->enc_U[1], &m->att_Wc, &m->init_W, &m->g1, &m->att_Wq, &m->g2,
                    &m->ro, &m->out})
    f.push_back(&P->d);
  if (m->precomp)
    for (Packed* P : {&m->g1x, &m->roy, &m->cpw}) f.push_back(&P->d);
  for (float** b : {&m->enc_in_b, &m->att_b, &m->init_b, &m->att_v, &m->ro_b}) f.push_back((void**)b);
  for (GruBias* g : {&m->enc_bias, &m->g1_bias, &m->g2_bias}) {
    f.push_back((void**)&g->brz);
    f.push_back((void**)&g->bni);
    f.push_back((void**)&g->bns);
  }
  return f;
}

static bool same_layout(const nmt_model* a, const nmt_model* b) {
  return memcmp(&a->dims, &b->dims, sizeof(nmt_dims)) == 0 && a->device == b->device && a->kc == b->kc &&
         a->emb_ld == b->emb_ld && a->mem.bytes == b->mem.bytes && a->mem.kind == b->mem.kind;
}

nmt_status nmt_model_average(int32_t K, nmt_model* const* models, const float* h_coef, void* stream,
                             nmt_model** out) {
  if (!out) return fail(NMT_EINVAL, "NULL argument");
  *out = nullptr;
  if (K < 1 || K > kMaxModels) return fail(NMT_ERANGE, "K must be in [1, %d] (got %d)", kMaxModels, K);
  if (!models) return fail(NMT_EINVAL, "NULL argument");
  for (int k = 0; k < K; ++k) {
    if (!models[k]) return fail(NMT_EINVAL, "models[%d] is NULL", k);
    if (!same_layout(models[0], models[k]))
      return fail(NMT_EINVAL, "models[%d] differs from models[0] in dimensions, weight type or device", k);
  }
  ModelTable tab{};
  for (int k = 0; k < K; ++k) {
    tab.w[k] = h_coef ? h_coef[k] : 1.f / (float)K;
    if (!std::isfinite(tab.w[k])) return fail(NMT_EINVAL, "coefficient %d is not finite", k);
  }
  const nmt_model* m0 = models[0];
  nmt_status rc = check_device(m0);
  if (rc != NMT_OK) return rc;
  hipStream_t st = (hipStream_t)stream;

  // Same dimensions and packing as models[0], fresh parameter buffers.
  nmt_model* a = new nmt_model(*m0);
  a->mem = Allocs{};
  a->prof_events.clear();
  a->prof_on = false;
  a->prof_max = a->prof_used = 0;
  a->err = nullptr;
  std::unordered_map<void*, void*> remap;
  hipError_t e = hipSuccess;
  size_t n_param = 0;
  for (size_t i = 0; i < m0->mem.ptrs.size() && e == hipSuccess; ++i) {
    const uint8_t kind = m0->mem.kind[i];
    if (kind == kOther) continue;
    void* p = nullptr;
    e = a->mem.alloc(&p, m0->mem.bytes[i], kind);
    if (e != hipSuccess) break;
    remap[m0->mem.ptrs[i]] = p;
    ++n_param;
    for (int k = 0; k < K; ++k) tab.p[k] = models[k]->mem.ptrs[i];
    const int64_t n = (int64_t)(m0->mem.bytes[i] / (kind == kParamBF16 ? 2 : 4));
    e = launch_average(K, n, tab, kind, a->bf16, p, st);
  }
  if (e == hipSuccess) {
    // every parameter field must move to a buffer of its own
    const std::vector<void**> fields = param_fields(a);
    bool complete = fields.size() == n_param;
    for (void** f : fields) {
      auto it = remap.find(*f);
      if (it == remap.end()) {
        complete = false;
        break;
      }
      *f = it->second;
    }
    if (!complete) {
      (void)hipStreamSynchronize(st);
      a->mem.release();
      delete a;
      return fail(NMT_EDEVICE, "nmt_model_average: parameter table does not match the model's buffers");
    }
    // the tables are products of the weights, not averaged: rebuilt from the averages
    a->tab_x = a->tab_y = nullptr;
    if (a->precomp) e = word_tables(a, st);
    if (e == hipSuccess) e = a->mem.alloc((void**)&a->err, sizeof(int));
  }
  if (e == hipSuccess) e = hipMemsetAsync(a->err, 0, sizeof(int), st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) {
    (void)hipStreamSynchronize(st);
    a->mem.release();
    delete a;
    return hip_fail(e, "nmt_model_average");
  }
  *out = a;
  return ok();
}

// Bytes an ensemble step of B rows actually uses: the models run one after
// another on the same workspace, so the largest single step.
static size_t ensemble_need(int32_t K, nmt_model* const* models, int32_t B) {
  size_t mx = 0;
  for (int k = 0; k < K; ++k) {
    const size_t b = ws_layout(models[k], B).total;
    mx = b > mx ? b : mx;
  }
  return mx;
}

// The largest nmt_score_workspace_bytes over the models, so that (as for one
// model) a workspace sized for B serves every smaller batch.
size_t nmt_ensemble_workspace_bytes(int32_t K, nmt_model* const* models, int32_t B) {
  if (!models || K < 1 || K > kMaxModels || B <= 0) return 0;
  size_t mx = 0;
  for (int k = 0; k < K; ++k) {
    if (!models[k]) return 0;
    const size_t b = nmt_score_workspace_bytes(models[k], B);
    mx = b > mx ? b : mx;
  }
  return mx;
}

nmt_status nmt_score_ensemble(int32_t K, nmt_model* const* models, const nmt_source* const* srcs, int32_t B,
                              const float* const* d_s_prev, const int32_t* d_y_prev, const int32_t* d_sent_id,
                              const int32_t* d_req, float* d_logp, float* const* d_s_new, float* d_logZ,
                              const float* h_weights, float* d_score, void* d_workspace, size_t ws_bytes,
                              void* stream) {
  if (K < 1 || K > kMaxModels) return fail(NMT_ERANGE, "K must be in [1, %d] (got %d)", kMaxModels, K);
  if (!models || !srcs || !d_s_prev || !d_s_new) return fail(NMT_EINVAL, "NULL argument");
  if (B < 0) return fail(NMT_EINVAL, "B must be >= 0 (got %d)", B);
  for (int k = 0; k < K; ++k) {
    if (!models[k] || !srcs[k]) return fail(NMT_EINVAL, "model or source %d is NULL", k);
    if (models[k]->dims.V != models[0]->dims.V || models[k]->device != models[0]->device)
      return fail(NMT_EINVAL, "model %d has another target vocabulary or device", k);
    if (srcs[k]->S != srcs[0]->S) return fail(NMT_EINVAL, "source %d holds another number of sentences", k);
    if (B > 0 && (!d_s_prev[k] || !d_s_new[k])) return fail(NMT_EINVAL, "state pointers of model %d are NULL", k);
  }
  if (B == 0) return ok();
  if (!d_y_prev || !d_sent_id || !d_req || !d_logp) return fail(NMT_EINVAL, "a required device pointer is NULL");
  ModelTable tab{};
  for (int k = 0; k < K; ++k) {
    tab.w[k] = h_weights ? h_weights[k] : 1.f;
    if (!std::isfinite(tab.w[k])) return fail(NMT_EINVAL, "weight %d is not finite", k);
  }
  // validate everything before the first launch: a failed call enqueues nothing
  const size_t need = ensemble_need(K, models, B);
  if (!d_workspace || ((uintptr_t)d_workspace & 255)) return fail(NMT_EINVAL, "workspace must be 256-byte aligned");
  if (ws_bytes < need) return fail(NMT_EWORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, need);
  for (int k = 0; k < K; ++k)
    if (!aligned16(d_s_prev[k]) || !aligned16(d_s_new[k]))
      return fail(NMT_EINVAL, "state arrays of model %d must be 16-byte aligned", k);
  nmt_status rc0 = check_device(models[0]);
  if (rc0 != NMT_OK) return rc0;
  for (int k = 0; k < K; ++k) {
    // one step per model on the caller's stream; the workspace is reused in stream order
    const nmt_status rc = nmt_score_batch(models[k], srcs[k], B, d_s_prev[k], d_y_prev, d_sent_id, d_req,
                                          d_logp + (int64_t)k * B, d_s_new[k],
                                          d_logZ ? d_logZ + (int64_t)k * B : nullptr, d_workspace, ws_bytes, stream);
    if (rc != NMT_OK) return rc;
  }
  if (d_score) {
    const hipError_t e = launch_weighted_sum(K, B, d_logp, tab, d_score, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "nmt_score_ensemble");
  }
  return ok();
}

}  // extern "C"

// Entry points for forest.hip.
namespace nmt {
nmt_status forest_fail(nmt_status st, const char* msg) { return fail(st, "%s", msg); }
}  // namespace nmt

nmt_status nmt_internal_score_step(nmt_model* m, const nmt_source* src, int32_t B, const float* pool,
                                   int32_t pool_rows, const int32_t* state_row, const int32_t* y_prev,
                                   const int32_t* sent_id, const int32_t* req_off, const int32_t* req, int32_t nreq,
                                   float* logp, float* s_new, void* ws, size_t ws_bytes, hipStream_t st,
                                   const AttnGroups* grp) {
  if (B == 0) return ok();
  Requests rq{req_off, req, nreq, state_row, pool_rows};
  return score_step(m, src, B, pool, pool_rows, state_row, y_prev, sent_id, rq, logp, s_new, nullptr, ws, ws_bytes, st,
                    nullptr, nullptr, nullptr, nullptr, grp);
}

// The attention grouping of several batches over one source in one launch
// (the levels of a forest): sets each level's rows per tile; false where the
// attention would not use a grouping (too many sentences), so the levels
// take the per-row kernel as single steps do.
bool nmt_internal_group_levels(const nmt_model* m, const nmt_source* src, GroupLevel* lv, int n, hipStream_t st,
                               hipError_t* err) {
  *err = hipSuccess;
  if (src->S > kGroupMaxS || src->Tpad > kMaxTpad) return false;
  for (int i = 0; i < n; ++i) lv[i].G = attn_rows_per_tile(lv[i].B, m->cus);
  *err = launch_group_levels(lv, n, src->S, src->len, src->Tpad, st);
  return *err == hipSuccess;
}

int32_t nmt_internal_hidden(const nmt_model* m) { return m->dims.H; }
int32_t nmt_internal_sentences(const nmt_source* src) { return src->S; }
int32_t nmt_internal_vocab(const nmt_model* m) { return m->dims.V; }
int nmt_internal_device(const nmt_model* m) { return m->device; }

extern "C" {

nmt_status nmt_stream_status(nmt_model* m, void* stream) {
  if (!m) return fail(NMT_EINVAL, "NULL model");
  nmt_status rc = check_device(m);
  if (rc != NMT_OK) return rc;
  hipError_t e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "nmt_stream_status");
  int flag = 0;
  e = hipMemcpy(&flag, m->err, sizeof(int), hipMemcpyDeviceToHost);
  if (e == hipSuccess && flag) e = hipMemset(m->err, 0, sizeof(int));
  if (e != hipSuccess) return hip_fail(e, "nmt_stream_status");
  if (flag) return fail(NMT_ERANGE, "an id was out of range in a call since the last status check");
  return ok();
}

}  // extern "C"

extern "C" {

nmt_status nmt_profile_begin(nmt_model* m, int32_t max_steps) {
  if (!m || max_steps < 1) return fail(NMT_EINVAL, "NULL model or max_steps < 1");
  nmt_status rc = check_device(m);
  if (rc != NMT_OK) return rc;
  (void)hipDeviceSynchronize();
  drop_profile_events(m);
  const size_t n = (size_t)max_steps * (NMT_NUM_PHASES + 1);
  m->prof_events.reserve(n);
  // Timing-only events: without the system-scope fence a recorded event
  // would otherwise add (an L2 write-back and invalidate), so the kernel
  // after each event runs as it does in an untimed step.
  for (size_t i = 0; i < n; ++i) {
    hipEvent_t ev;
    hipError_t e = hipEventCreateWithFlags(&ev, hipEventDisableSystemFence);
    if (e != hipSuccess) {
      drop_profile_events(m);
      return hip_fail(e, "nmt_profile_begin");
    }
    m->prof_events.push_back(ev);
  }
  m->prof_max = max_steps;
  m->prof_used = 0;
  m->prof_on = true;
  return ok();
}

nmt_status nmt_profile_end(nmt_model* m, void* stream, nmt_timing* out) {
  if (!m || !out) return fail(NMT_EINVAL, "NULL model or output");
  if (!m->prof_on) return fail(NMT_EINVAL, "no profile is running");
  hipError_t e = hipStreamSynchronize((hipStream_t)stream);
  nmt_timing t{};
  t.steps = m->prof_used;
  for (int s = 0; s < m->prof_used && e == hipSuccess; ++s) {
    hipEvent_t* ev = &m->prof_events[(size_t)s * (NMT_NUM_PHASES + 1)];
    for (int p = 0; p < NMT_NUM_PHASES && e == hipSuccess; ++p) {
      float ms = 0.f;
      e = hipEventElapsedTime(&ms, ev[p], ev[p + 1]);
      t.ms[p] += ms;
    }
  }
  drop_profile_events(m);
  if (e != hipSuccess) return hip_fail(e, "nmt_profile_end");
  *out = t;
  return ok();
}

}  // extern "C"
