// device.hpp -- shared device-side building blocks of libnmt (gfx950 only).
//
// GEMM tiles follow one scheme everywhere.  A workgroup owns a TM x TN
// output tile and walks K in chunks of KC, double-buffered in LDS.
//
//  * A operand (activations): up to three row-major fp32 segments that are
//    concatenated along K without being materialised (for example
//    [embedding rows gathered by word id | previous state]).  Each segment
//    is read in float4 pieces; a segment's K is padded up to KC with zeros.
//  * B operand (weights): packed once at model creation into
//    [Kpad/4][Npad][4] ("k4-interleaved"), so one float4 holds four
//    consecutive k of one output column.
//  * MFMA: v_mfma_f32_32x32x2f32.  Lane l of a wave supplies A[l%32][k] and
//    B[k][l%32] with k = l/32.  Within a group of 8 k values, lane half h
//    uses k = 4h + j on the j-th of four MFMAs, so each lane reads exactly
//    one float4 of A and one of B per four MFMAs (ds_read_b128).  The sum
//    over k is order-free, so this permutation changes nothing but the
//    rounding order.
//  * Accumulator layout (checked on the device): register r of lane l
//    holds row 8*(r/4) + 4*(l/32) + r%4 and column l%32 of the 32x32 block.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace nmt {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;

// One A-operand segment.
struct ASeg {
  const float* p;         // row-major fp32 matrix
  const int32_t* gather;  // nullable: row m reads row gather[m] of p; ids outside [0, gmax) read zeros
  int32_t gmax;           // rows of p addressable through gather
  int64_t ld;             // row stride in floats (multiple of 4)
  int32_t K;              // valid columns (multiple of 4)
  int32_t nchunk;         // ceil(K / KC)
  int32_t side;           // 0: input side, 1: state side (routes the GRU candidate gate)
};

struct AOperand {
  ASeg seg[3];
  int32_t nseg;
  int32_t M;  // valid rows
};

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

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
  return s;
}

__device__ __forceinline__ int total_chunks(const AOperand& A) {
  return (A.nseg > 0 ? A.seg[0].nchunk : 0) + (A.nseg > 1 ? A.seg[1].nchunk : 0) +
         (A.nseg > 2 ? A.seg[2].nchunk : 0);
}

__device__ __forceinline__ const float* seg_row(const ASeg& s, int row, int M) {
  if (row >= M) return nullptr;
  if (s.gather) {
    int g = s.gather[row];
    if (g < 0 || g >= s.gmax) return nullptr;
    return s.p + (int64_t)g * s.ld;
  }
  return s.p + (int64_t)row * s.ld;
}

// Global -> register -> LDS staging of one K chunk of the A and B tiles.
// Each thread owns one tile row for A (NT % TM == 0) and strided float4s of B.
template <int TM, int TN, int KC, int NT>
struct Stager {
  static constexpr int KQ = KC / 4;
  static constexpr int NA = TM * KQ / NT;
  static constexpr int NB = TN * KQ / NT;
  static_assert(NT % TM == 0, "one A row per thread");
  static_assert((TM * KQ) % NT == 0 && (TN * KQ) % NT == 0, "whole float4s per thread");
  f32x4 ra[NA];
  f32x4 rb[NB];

  // arow: this thread's row of the current segment (nullptr = zeros);
  // kseg: k offset of the chunk within the segment; kq_glob: chunk start in
  // packed-weight rows of 4.
  __device__ __forceinline__ void load(const float* arow, int segK, int kseg, const float* __restrict__ Wp,
                                       int64_t Npad, int64_t kq_glob, int n0) {
    const int tid = threadIdx.x;
    const int kq0 = tid / TM;
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      int k = kseg + 4 * (kq0 + i * (NT / TM));
      ra[i] = (arow && k < segK) ? *(const f32x4*)(arow + k) : zero4();
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      int idx = tid + i * NT;
      int n = idx % TN, kq = idx / TN;
      rb[i] = *(const f32x4*)(Wp + ((kq_glob + kq) * Npad + n0 + n) * 4);
    }
  }

  __device__ __forceinline__ void store(float* As, float* Bs) const {
    const int tid = threadIdx.x;
    const int m = tid % TM, kq0 = tid / TM;
#pragma unroll
    for (int i = 0; i < NA; ++i) *(f32x4*)(As + ((kq0 + i * (NT / TM)) * TM + m) * 4) = ra[i];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      int idx = tid + i * NT;
      int n = idx % TN, kq = idx / TN;
      *(f32x4*)(Bs + (kq * TN + n) * 4) = rb[i];
    }
  }
};

__device__ __forceinline__ f32x16 mfma(float a, float b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// Fragment loads from the staged LDS tiles: the float4 for k group kg of the
// 32-row (or 32-column) block starting at r0.
template <int TROWS>
__device__ __forceinline__ f32x4 lds_frag(const float* S, int kg, int r0) {
  const int lane = threadIdx.x & 63;
  return *(const f32x4*)(S + ((2 * kg + (lane >> 5)) * TROWS + r0 + (lane & 31)) * 4);
}

// The generic main loop: walks chunks [c_begin, c_end) of the A segments
// (all chunks by default), staging the next chunk while
// `compute(As, Bs, side)` runs on the current one.  Chunk c covers packed
// weight rows c*KC .. c*KC+KC-1, whichever segment it falls in.
template <int TM, int TN, int KC, int NT, class Compute>
__device__ __forceinline__ void gemm_mainloop(const AOperand& A, const float* __restrict__ Wp, int64_t Npad,
                                              int m0, int n0, float* lds, Compute&& compute, int c_begin = 0,
                                              int c_end = 1 << 30) {
  constexpr int ASZ = TM * KC, BSZ = TN * KC;
  float* As[2] = {lds, lds + ASZ + BSZ};
  float* Bs[2] = {lds + ASZ, lds + 2 * ASZ + BSZ};
  Stager<TM, TN, KC, NT> st;
  const int row = m0 + (int)threadIdx.x % TM;

  const int nc = total_chunks(A);
  if (c_end > nc) c_end = nc;
  if (c_begin >= c_end) return;

  int seg = 0, ch = c_begin;
  ASeg sg = seg_at(A, 0);
  while (ch >= sg.nchunk) {
    ch -= sg.nchunk;
    sg = seg_at(A, ++seg);
  }
  const float* arow = seg_row(sg, row, A.M);
  st.load(arow, sg.K, ch * KC, Wp, Npad, (int64_t)c_begin * (KC / 4), n0);
  st.store(As[0], Bs[0]);
  __syncthreads();

  for (int c = c_begin; c < c_end; ++c) {
    const bool more = c + 1 < c_end;
    const int buf = (c - c_begin) & 1;
    const int side = sg.side;
    if (more) {
      if (++ch == sg.nchunk) {
        ch = 0;
        do { sg = seg_at(A, ++seg); } while (sg.nchunk == 0);
        arow = seg_row(sg, row, A.M);
      }
      st.load(arow, sg.K, ch * KC, Wp, Npad, (int64_t)(c + 1) * (KC / 4), n0);
    }
    compute(As[buf], Bs[buf], side);
    if (more) st.store(As[buf ^ 1], Bs[buf ^ 1]);
    __syncthreads();
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

__device__ __forceinline__ float sigmoidf_(float x) { return 1.f / (1.f + expf(-x)); }

// Row of accumulator register r for lane half h.
__device__ __forceinline__ int acc_row(int r, int h) { return 8 * (r >> 2) + 4 * h + (r & 3); }

}  // namespace nmt
