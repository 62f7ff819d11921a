// device.hpp -- shared device-side building blocks of libnmt (gfx950 only).
//
// GEMM tiles follow one scheme in both precisions.  The unit of data is a
// 16-byte vector holding KV consecutive k of one row (A) or one column (B):
// four fp32 (KV = 4) or eight bf16 (KV = 8).
//
//  * A operand (activations): up to three row-major segments concatenated
//    along K without being materialised (for example [embedding rows
//    gathered by word id | previous state]).  Segments are fp32, or bf16
//    for embedding tables stored in bf16 (rows padded to whole vectors).
//    The bf16 path rounds fp32 activations to bf16 (nearest even) as it
//    stages them; accumulation is always fp32.
//  * B operand (weights): packed once at model creation into
//    [Kpad/KV][Npad][KV], so one 16-byte load fetches a whole vector.
//  * A workgroup owns a TM x TN output tile and walks K in chunks of
//    KC = KQ * KV (KQ vectors per row per chunk), double-buffered in LDS laid
//    out as [KQ][rows][16 B].
//  * MFMA: lane l of a wave supplies row (or column) l%32; lane half
//    h = l/32 supplies vector 2*kg + h of k group kg.  fp32 issues four
//    v_mfma_f32_32x32x2f32 per vector pair (k = 4h + j on the j-th);
//    bf16 issues one v_mfma_f32_32x32x16_bf16 (k = 8h + e).  The sum over
//    k is order-free, so this only fixes the rounding order.
//  * Accumulator layout (checked on the device): register r of lane l
//    holds row 8*(r/4) + 4*(l/32) + r%4 and column l%32 of the 32x32 block.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

namespace nmt {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// f(std::integral_constant<int, i>{}) for i = 0 .. N-1, unrolled at compile time.
template <int N, class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl<N>(f, std::make_integer_sequence<int, N>{});
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// Eight floats rounded to bf16 (nearest even), returned as 16 raw bytes.
__device__ __forceinline__ f32x4 pack_bf16(const f32x4& x0, const f32x4& x1) {
  bf16x8 v;
  v[0] = (__bf16)x0[0];
  v[1] = (__bf16)x0[1];
  v[2] = (__bf16)x0[2];
  v[3] = (__bf16)x0[3];
  v[4] = (__bf16)x1[0];
  v[5] = (__bf16)x1[1];
  v[6] = (__bf16)x1[2];
  v[7] = (__bf16)x1[3];
  return __builtin_bit_cast(f32x4, v);
}

// Vectors per row per K chunk of the LDS-staged GEMM tiles, per precision.
#ifndef NMT_KQ_F32
#define NMT_KQ_F32 8
#endif
#ifndef NMT_KQ_BF16
#define NMT_KQ_BF16 8
#endif

struct PrecF32 {
  static constexpr bool kBF16 = false;
  static constexpr int KV = 4;           // k per 16-byte vector
  static constexpr int KQ = NMT_KQ_F32;  // vectors per row per chunk
  static constexpr int KC = KQ * KV;     // k per chunk
  __device__ static __forceinline__ void mma(const f32x4& a, const f32x4& b, f32x16& acc) {
#pragma unroll
    for (int j = 0; j < 4; ++j) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[j], b[j], acc, 0, 0, 0);
  }
  // a*b with a zero accumulator (encoded as an inline constant, no clearing moves)
  __device__ static __forceinline__ f32x16 mma0(const f32x4& a, const f32x4& b) {
    f32x16 acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0], b[0], f32x16{}, 0, 0, 0);
#pragma unroll
    for (int j = 1; j < 4; ++j) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[j], b[j], acc, 0, 0, 0);
    return acc;
  }
};

struct PrecBF16 {
  static constexpr bool kBF16 = true;
  static constexpr int KV = 8;
  static constexpr int KQ = NMT_KQ_BF16;
  static constexpr int KC = KQ * KV;
  __device__ static __forceinline__ void mma(const f32x4& a, const f32x4& b, f32x16& acc) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), acc,
                                                  0, 0, 0);
  }
  __device__ static __forceinline__ f32x16 mma0(const f32x4& a, const f32x4& b) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                   f32x16{}, 0, 0, 0);
  }
};

// One A-operand segment.
struct ASeg {
  const void* p;          // row-major matrix, fp32 or (bf16 = 1) bf16
  const int32_t* gather;  // nullable: row m reads row gather[m] of p; ids outside [0, gmax) read zeros
  int32_t gmax;           // rows of p addressable through gather
  int64_t ld;             // row stride in elements (bf16 rows: a multiple of 8, zero-padded)
  int32_t K;              // valid columns (fp32: a multiple of 4; bf16: the padded row length)
  int32_t nchunk;         // ceil(K / KC)
  int32_t side;           // 0: input side, 1: state side (routes the GRU candidate gate)
  int32_t bf16;           // element type of p
};

struct AOperand {
  ASeg seg[3];
  int32_t nseg;
  int32_t M;  // valid rows
};

// Segment i of A, field by field through uniform selects: indexing the
// by-value kernel argument (or copying whole segments conditionally) with a
// runtime index makes the compiler spill it to scratch memory.
template <class T>
__device__ __forceinline__ T sel3(int i, T a, T b, T c) {
  return i == 0 ? a : (i == 1 ? b : c);
}
__device__ __forceinline__ ASeg seg_at(const AOperand& A, int i) {
  ASeg s;
  s.p = sel3(i, A.seg[0].p, A.seg[1].p, A.seg[2].p);
  s.gather = sel3(i, A.seg[0].gather, A.seg[1].gather, A.seg[2].gather);
  s.gmax = sel3(i, A.seg[0].gmax, A.seg[1].gmax, A.seg[2].gmax);
  s.ld = sel3(i, A.seg[0].ld, A.seg[1].ld, A.seg[2].ld);
  s.K = sel3(i, A.seg[0].K, A.seg[1].K, A.seg[2].K);
  s.nchunk = sel3(i, A.seg[0].nchunk, A.seg[1].nchunk, A.seg[2].nchunk);
  s.side = sel3(i, A.seg[0].side, A.seg[1].side, A.seg[2].side);
  s.bf16 = sel3(i, A.seg[0].bf16, A.seg[1].bf16, A.seg[2].bf16);
  return s;
}

__device__ __forceinline__ int total_chunks(const AOperand& A) {
  return (A.nseg > 0 ? A.seg[0].nchunk : 0) + (A.nseg > 1 ? A.seg[1].nchunk : 0) +
         (A.nseg > 2 ? A.seg[2].nchunk : 0);
}

// Raw buffer resource over `bytes` bytes at p.  The GEMM staging reads
// through such resources with a per-lane byte offset and a per-chunk scalar
// offset; a lane offset of kNoLoad is past every resource (all of them stay
// under 2 GiB, checked on the host), so that load reads zeros without
// touching memory.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* p, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)p, (short)0, (int)bytes, 0x00020000);
}
constexpr int kNoLoad = (int)0x80000000u;
__device__ __forceinline__ f32x4 buf_load(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// Bytes of the matrix behind segment s (M rows, or gmax rows if gathered).
__device__ __forceinline__ int64_t seg_bytes(const ASeg& s, int M) {
  return (int64_t)(s.gather ? s.gmax : M) * s.ld * (s.bf16 ? 2 : 4);
}

// Byte offset of this thread's row of segment s, or kNoLoad for a row past
// M or an out-of-range id (a zero row).
__device__ __forceinline__ int seg_row_off(const ASeg& s, int row, int M) {
  if (row >= M) return kNoLoad;
  int r = row;
  if (s.gather) {
    r = s.gather[row];
    if (r < 0 || r >= s.gmax) return kNoLoad;
  }
  return (int)((int64_t)r * s.ld * (s.bf16 ? 2 : 4));
}

// The raw data behind one A vector for the staging: one 16-byte load (fp32,
// or a bf16 source whose rows are padded to whole vectors) or, for bf16 from
// an fp32 source, two.  `roff` is the row's byte offset, `k` the vector's
// column and `soff` the chunk's scalar byte offset (its column times the
// element size, already part of k).  Absent rows and columns read zeros.
// Every call issues the same loads whatever the data, so the compiler can
// count the loads in flight exactly, and nothing consumes the values until
// they are stored to LDS.
template <class P, bool SRC16>
__device__ __forceinline__ void load_a_raw(__amdgpu_buffer_rsrc_t res, int roff, int K, int k, int kin, int soff,
                                           f32x4& x0, f32x4& x1) {
  // kin: the vector's column within the chunk (k = chunk column + kin)
  const int o = roff + kin * (P::kBF16 && SRC16 ? 2 : 4);
  x0 = buf_load(res, k < K ? o : kNoLoad, soff);
  if constexpr (P::kBF16 && !SRC16) x1 = buf_load(res, k + 4 < K ? o + 16 : kNoLoad, soff);
}

// The A vector from load_a_raw's data, in precision P.
template <class P, bool SRC16>
__device__ __forceinline__ f32x4 a_from_raw(const f32x4& x0, const f32x4& x1) {
  if constexpr (P::kBF16 && !SRC16) return pack_bf16(x0, x1);
  return x0;
}

// The 16-byte A vector at column k of a row, in precision P.
template <class P>
__device__ __forceinline__ f32x4 load_a_vec(const char* row, int bf16src, int K, int k) {
  if (!row || k >= K) return zero4();
  if constexpr (P::kBF16) {
    if (bf16src) return *(const f32x4*)(row + 2 * (int64_t)k);  // rows padded to whole vectors
    const float* r = (const float*)row;
    const f32x4 x0 = *(const f32x4*)(r + k);
    const f32x4 x1 = k + 4 < K ? *(const f32x4*)(r + k + 4) : zero4();
    return pack_bf16(x0, x1);
  } else {
    return *(const f32x4*)((const float*)row + k);
  }
}

// Vector kq of an activation row with 1 at the bias slots k = E .. E+nb-1
// (the output weights carry the bias in those rows).
template <class P>
__device__ __forceinline__ f32x4 with_bias_ones(f32x4 v, int kq, int E, int nb) {
  const int k0 = kq * P::KV;
  if (k0 + P::KV <= E || k0 >= E + nb) return v;
  // slots past E: 1 at the bias slots, 0 after them (whatever the row's
  // memory held there)
  if constexpr (P::kBF16) {
    bf16x8 b = __builtin_bit_cast(bf16x8, v);
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (k0 + e >= E) b[e] = (__bf16)(k0 + e < E + nb ? 1.f : 0.f);
    return __builtin_bit_cast(f32x4, b);
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (k0 + e >= E) v[e] = k0 + e < E + nb ? 1.f : 0.f;
    return v;
  }
}

// An A stage in LDS is [KQ][a_rows] vectors.  The staging stores are
// transposed (consecutive lanes write consecutive vectors of one row, a
// stage row apart), which would put them all in the same banks.  fp32 pads
// each vector's rows by one vector; bf16 keeps row r of vector v at row
// r ^ a_swz(v), a permutation within each aligned block of 32 rows, so a
// fragment's 32 rows stay 32 distinct slots (measured: the swizzle is a
// little faster for the bf16 GRU tile, the padding for the fp32 one, whose
// fragment reads then need no address arithmetic).
template <int TM, class P>
constexpr int a_rows() {
  return P::kBF16 ? TM : TM + 1;
}
template <class P>
__device__ __forceinline__ int a_swz(int v) {
  return P::kBF16 ? (v & (P::KQ - 1) & 31) : 0;
}

// Global -> register -> LDS staging of one K chunk of the A and B tiles.
// Vector v of the chunk's TM x KQ A vectors is row v / KQ, vector v % KQ, so
// consecutive lanes read consecutive 16-byte pieces of one row (KQ lanes per
// row: one contiguous 128-byte fp32 or 256-byte bf16-from-fp32 stretch).
// B vectors are consecutive columns of one packed row.
// SRC16: the A segment is stored in bf16 (only with bf16 weights).
template <int TM, int TN, int NT, class P, bool SRC16>
struct Stager {
  static constexpr int KQ = P::KQ;
  static constexpr int NA = TM * KQ / NT;
  static constexpr int NB = TN * KQ / NT;
  static_assert((TM * KQ) % NT == 0 && (TN * KQ) % NT == 0, "whole vectors per thread");
  static constexpr bool kTwo = P::kBF16 && !SRC16;  // bf16 from an fp32 source: two raw vectors
  f32x4 ra[NA], rx[kTwo ? NA : 1];
  f32x4 rb[NB];

  // Tile row of this thread's i-th A vector (the rows it reads: see rows()).
  __device__ static __forceinline__ int a_row(int i) { return ((int)threadIdx.x + i * NT) / KQ; }
  __device__ static __forceinline__ int a_vec(int i) { return ((int)threadIdx.x + i * NT) % KQ; }

  // aoff[i]: byte offset of the row of this thread's i-th A vector in the
  // segment's resource; kseg: k offset of the chunk within the segment;
  // bvo[i]: byte offset of its i-th B vector within a chunk of the packed
  // weights, whose chunk starts at scalar offset bsoff.  Weights first:
  // their loads carry no condition.
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t ares, const int (&aoff)[NA], int segK, int kseg,
                                       __amdgpu_buffer_rsrc_t bres, const int (&bvo)[NB], int bsoff) {
#pragma unroll
    for (int i = 0; i < NB; ++i) rb[i] = buf_load(bres, bvo[i], bsoff);
    const int asoff = kseg * (P::kBF16 && SRC16 ? 2 : 4);
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      f32x4 x1;
      const int kin = P::KV * a_vec(i);
      load_a_raw<P, SRC16>(ares, aoff[i], segK, kseg + kin, kin, asoff, ra[i], x1);
      if constexpr (kTwo) rx[i] = x1;
    }
  }

  // Byte offset of this thread's i-th B vector within a chunk.
  __device__ static __forceinline__ int b_off(int i, int64_t Npad, int n0) {
    const int idx = (int)threadIdx.x + i * NT;
    const int n = idx % TN, kq = idx / TN;
    return (int)(((int64_t)kq * Npad + n0 + n) * 16);
  }

  __device__ __forceinline__ void store(f32x4* As, f32x4* Bs) const {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < NA; ++i)
      As[a_vec(i) * a_rows<TM, P>() + (a_row(i) ^ a_swz<P>(a_vec(i)))] = a_from_raw<P, SRC16>(ra[i], rx[kTwo ? i : 0]);
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int idx = tid + i * NT;
      const int n = idx % TN, kq = idx / TN;
      Bs[kq * TN + n] = rb[i];
    }
  }
};

// Fragment of k group kg for the 32-row (or 32-column) block at r0.
template <int TROWS>
__device__ __forceinline__ f32x4 lds_frag(const f32x4* S, int kg, int r0) {
  const int lane = threadIdx.x & 63;
  return S[(2 * kg + (lane >> 5)) * TROWS + r0 + (lane & 31)];
}
// The same from an A stage of TM rows (padded or swizzled: a_rows, a_swz).
template <int TM, class P>
__device__ __forceinline__ f32x4 lds_frag_a(const f32x4* S, int kg, int r0) {
  const int lane = threadIdx.x & 63, v = 2 * kg + (lane >> 5);
  return S[v * a_rows<TM, P>() + r0 + ((lane & 31) ^ a_swz<P>(v))];
}

// Global-load lookahead of the tile GEMMs: chunks whose loads are in
// flight in registers while a chunk is computed from LDS (the GRU tile; the
// plain tiles use NMT_PLAIN_LA).
#ifndef NMT_GEMM_LA
#define NMT_GEMM_LA 2
#endif
#ifndef NMT_GEMM_LA_BF16
#define NMT_GEMM_LA_BF16 2
#endif
#ifndef NMT_PLAIN_LA
#define NMT_PLAIN_LA 2
#endif
#ifndef NMT_PLAIN_LA_BF16
#define NMT_PLAIN_LA_BF16 2
#endif
template <class P>
constexpr int kGruLA = P::kBF16 ? NMT_GEMM_LA_BF16 : NMT_GEMM_LA;
template <class P>
constexpr int kPlainLA = P::kBF16 ? NMT_PLAIN_LA_BF16 : NMT_PLAIN_LA;

// MFMAs issued between two staging loads (measured: fp32 1, bf16 2).
#ifndef NMT_GEMM_MFMA_PER_LOAD_F32
#define NMT_GEMM_MFMA_PER_LOAD_F32 1
#endif
#ifndef NMT_GEMM_MFMA_PER_LOAD_BF16
#define NMT_GEMM_MFMA_PER_LOAD_BF16 2
#endif
template <class P>
constexpr int kMfmaPerLoad = P::kBF16 ? NMT_GEMM_MFMA_PER_LOAD_BF16 : NMT_GEMM_MFMA_PER_LOAD_F32;

// Work of one k group of a wave's compute: kFrags fragment reads from LDS
// and kMfma MFMAs.
template <int FR, int MK>
struct KgShape {
  static constexpr int kFrags = FR, kMfma = MK;
};

// Instruction order of one chunk step with NL staging loads: the first k
// group's fragment reads, then per k group one MFMA, the next k group's
// fragment reads (so they land while this group's MFMAs run), and the rest
// of the group's MFMAs with the step's loads spread among them.
template <class KS, int NKG, int NL>
__device__ __forceinline__ void sched_chunk_step() {
  constexpr int FR = KS::kFrags, MK = KS::kMfma;
  __builtin_amdgcn_sched_group_barrier(0x100, FR, 0);
  static_for<NKG>([&](auto kc) {
    constexpr int kg = decltype(kc)::value;
    constexpr int nl = (kg + 1) * NL / NKG - kg * NL / NKG;  // loads placed in this k group
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if constexpr (kg + 1 < NKG) __builtin_amdgcn_sched_group_barrier(0x100, FR, 0);
    static_for<nl>([&](auto lc) {
      constexpr int l = decltype(lc)::value;
      constexpr int before = (l + 1) * (MK - 1) / nl - l * (MK - 1) / nl;  // MFMAs ahead of load l
      if constexpr (before > 0) __builtin_amdgcn_sched_group_barrier(0x008, before, 0);
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    });
    if constexpr (nl == 0 && MK > 1) __builtin_amdgcn_sched_group_barrier(0x008, MK - 1, 0);
  });
}

// Main loop over chunks [cb, ce) of one A segment (chunk indices local to
// the segment; vq0 = packed weight vector row of the segment's chunk 0).
// KS (a KgShape, or void) describes the compute's k groups for the
// instruction order of a step (sched_chunk_step).
// Chunk i's global loads are issued LA iterations before it is computed
// (into register set i % LA), it is stored to LDS stage i % 2 at the end of
// iteration i - 1, and `compute(As, Bs)` runs on it at iteration i.  The
// loop is unrolled by LA so register sets are picked at compile time.  Ends
// with a barrier, so a following call may reuse the LDS stages.
template <int TM, int TN, int NT, class P, bool SRC16, int LA, class KS, class Compute>
__device__ __forceinline__ void gemm_segment_t(const ASeg& sg, int M, const f32x4* __restrict__ Wp, int64_t Npad,
                                               int m0, int n0, f32x4* lds, Compute&& compute, int64_t vq0, int cb,
                                               int ce) {
  // Stage s holds A at lds + s*STG and B right after it.  Stage bases are
  // formed as offsets from `lds` itself: a runtime-indexed array of stage
  // pointers hides the LDS address space from the compiler, which then emits
  // flat loads that share the global-load counter, so every fragment wait
  // would also wait for the next chunk's prefetch.
  constexpr int KQ = P::KQ;
  constexpr int ASZ = a_rows<TM, P>() * KQ, BSZ = TN * KQ, STG = ASZ + BSZ;  // vectors per stage
  using St = Stager<TM, TN, NT, P, SRC16>;
  const int n = ce - cb;
  if (n <= 0) return;
  St st[LA];
  // the segment's A rows and its packed weights (vector rows vq0 ..), each
  // through a buffer resource
  const __amdgpu_buffer_rsrc_t ares = buffer_rsrc(sg.p, seg_bytes(sg, M));
  const __amdgpu_buffer_rsrc_t bres = buffer_rsrc(Wp + vq0 * Npad, (int64_t)sg.nchunk * KQ * Npad * 16);
  int aoff[St::NA], bvo[St::NB];
#pragma unroll
  for (int i = 0; i < St::NA; ++i) aoff[i] = seg_row_off(sg, m0 + St::a_row(i), M);
#pragma unroll
  for (int i = 0; i < St::NB; ++i) bvo[i] = St::b_off(i, Npad, n0);
  // Loads are unconditional: past the segment's last chunk they re-read it,
  // so every iteration issues the same loads and the waits before the
  // stores count them exactly.
  auto load = [&](St& s, int i) {
    const int c = cb + (i < n ? i : n - 1);
    s.load(ares, aoff, sg.K, c * P::KC, bres, bvo, (int)((int64_t)c * KQ * Npad * 16));
  };
  static_for<LA>([&](auto j) { load(st[j], j); });
  st[0].store(lds, lds + ASZ);
  __syncthreads();
  // One step: chunk i's loads went out LA steps ago into register set j; it
  // is computed from LDS stage i % 2 while chunk i + 1 is stored to the
  // other stage.
  auto step = [&](int i, auto jc, bool store_next) {
    constexpr int j = decltype(jc)::value;  // this step's register set
    const int cur = (i & 1) * STG, nxt = STG - cur;
    load(st[j], i + LA);
    compute(lds + cur, lds + cur + ASZ);
    // The loads go out spread among the compute's MFMAs, so a load that
    // waits for the memory pipeline to take it (a chunk's loads are about
    // 56 KB per CU in bf16) does not hold up the matrix cores.  Left to the
    // scheduler, the loads sank below the compute and their registers were
    // reused by the fragment reads, whose writes then waited for the loads;
    // issued all before the compute, their issue stalled the wave for about
    // 480 cycles per chunk.  With a k-group shape KS, each k group's
    // fragment reads are also issued during the previous k group's MFMAs
    // (otherwise each read lands just before the MFMA that waits for it).
    if constexpr (!std::is_void_v<KS>) {
      sched_chunk_step<KS, P::KQ / 2, St::NB + St::NA * (St::kTwo ? 2 : 1)>();
    } else {
      static_for<St::NB + St::NA * (St::kTwo ? 2 : 1)>([&](auto) {
        __builtin_amdgcn_sched_group_barrier(0x008, kMfmaPerLoad<P>, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      });
    }
    if (store_next) st[(j + 1) % LA].store(lds + nxt, lds + nxt + ASZ);
    __syncthreads();
  };
  // Whole groups of LA steps with every store unconditional (the last step
  // of the segment stores a re-read chunk that nobody reads), so no path
  // round the loop skips the waits that retire a register set's loads; a
  // skipped store on such a path made the compiler wait for all loads in
  // flight at the top of every step.  The remaining steps follow.
  int i0 = 0;
  for (; i0 + LA <= n; i0 += LA) static_for<LA>([&](auto jc) { step(i0 + decltype(jc)::value, jc, true); });
  static_for<LA - 1>([&](auto jc) {
    const int i = i0 + decltype(jc)::value;
    if (i < n) step(i, jc, i + 1 < n);
  });
}

// gemm_segment_t with the segment's element type fixed at compile time (a
// runtime choice between the two load paths made the compiler issue both
// into the same registers, each waiting for the other).
template <int TM, int TN, int NT, class P, int LA = NMT_GEMM_LA, class KS = void, class Compute>
__device__ __forceinline__ void gemm_segment(const ASeg& sg, int M, const f32x4* __restrict__ Wp, int64_t Npad,
                                             int m0, int n0, f32x4* lds, Compute&& compute, int64_t vq0, int cb,
                                             int ce) {
  if constexpr (P::kBF16) {
    if (sg.bf16) {
      gemm_segment_t<TM, TN, NT, P, true, LA, KS>(sg, M, Wp, Npad, m0, n0, lds, compute, vq0, cb, ce);
      return;
    }
  }
  gemm_segment_t<TM, TN, NT, P, false, LA, KS>(sg, M, Wp, Npad, m0, n0, lds, compute, vq0, cb, ce);
}

// All segments of A, restricted to global chunks [c_begin, c_end) (chunk c
// covers packed weight vector rows KQ*c .. KQ*c+KQ-1, whichever segment it
// falls in).
template <int TM, int TN, int NT, class P, int LA = NMT_GEMM_LA, class KS = void, class Compute>
__device__ __forceinline__ void gemm_mainloop(const AOperand& A, const f32x4* __restrict__ Wp, int64_t Npad, int m0,
                                              int n0, f32x4* lds, Compute&& compute, int c_begin = 0,
                                              int c_end = 1 << 30) {
  int s0 = 0;
  for (int i = 0; i < A.nseg; ++i) {
    const ASeg sg = seg_at(A, i);
    const int s1 = s0 + sg.nchunk;
    const int cb = c_begin > s0 ? c_begin : s0, ce = c_end < s1 ? c_end : s1;
    gemm_segment<TM, TN, NT, P, LA, KS>(sg, A.M, Wp, Npad, m0, n0, lds, compute, (int64_t)s0 * P::KQ, cb - s0,
                                        ce - s0);
    s0 = s1;
  }
}

// Reductions within each 32-lane half of a wave (the lanes that share a
// row of an MFMA accumulator block).
__device__ __forceinline__ float half_max(float v) {
#pragma unroll
  for (int o = 16; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 32));
  return v;
}
__device__ __forceinline__ float half_sum(float v) {
#pragma unroll
  for (int o = 16; o >= 1; o >>= 1) v += __shfl_xor(v, o, 32);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// The cells' nonlinearities through the hardware's 2^x and reciprocal
// (about one ulp each) instead of the libm functions and an IEEE divide
// (some 80 instructions per GRU unit): sigma(x) = 1 / (1 + 2^{-x log2 e}),
// tanh(x) = 1 - 2 / (2^{2x log2 e} + 1).  Absolute error a few 1e-7; both
// saturate exactly (2^x overflows to inf, whose reciprocal is 0).
#ifndef NMT_FAST_CELL
#define NMT_FAST_CELL 1
#endif
__device__ __forceinline__ float sigmoidf_(float x) {
#if NMT_FAST_CELL
  return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-kLog2e * x));
#else
  return 1.f / (1.f + expf(-x));
#endif
}
__device__ __forceinline__ float tanhf_(float x) {
#if NMT_FAST_CELL
  return fmaf(-2.f, __builtin_amdgcn_rcpf(__builtin_amdgcn_exp2f(2.f * kLog2e * x) + 1.f), 1.f);
#else
  return tanhf(x);
#endif
}

// Row of accumulator register r for lane half h.
__device__ __forceinline__ int acc_row(int r, int h) { return 8 * (r >> 2) + 4 * h + (r & 3); }

}  // namespace nmt
