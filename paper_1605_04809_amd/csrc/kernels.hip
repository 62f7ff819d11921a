// kernels.hip -- the HIP kernels of one batched decoder step and of source
// initialisation, for gfx950.  Equations are listed in include/nmt.h.
// The GEMM-family kernels are templates over the precision policy
// (PrecF32: fp32 weights, PrecBF16: bf16 weights with bf16 MFMA inputs;
// both accumulate in fp32).
//
//   k_gemm_plain   MFMA GEMM with bias (+tanh) epilogue, optionally split
//                  over K: attention query, readout, attention keys,
//                  encoder input projections, initial state.
//   k_gemm_gru     MFMA GEMM whose tile holds matching r, z and candidate
//                  columns of the same hidden units, with the GRU cell fused
//                  into the epilogue (both decoder GRUs, encoder recurrence);
//                  128- or 64-row tiles by batch size.  Its SPLIT form sums
//                  a share of K and k_gru_cell adds the shares and applies
//                  the cell (the encoder's few-row recurrence).
//   k_vocab_lse    MFMA vocabulary projection streaming the output weights,
//                  fused with an online log-sum-exp; logits never reach HBM.
//   k_lse_combine  merges the per-slice partials, scores the requested word
//                  and checks the row's ids.
//   k_group_rows, k_attention_grouped
//                  masked MLP attention and context, rows grouped by
//                  sentence so a block reads each key and annotation once
//                  for several rows (k_attention: one row per block).
//   k_key_factors  the keys' factors 2^{2 log2(e) pctx} the attention
//                  scores read, and each sentence's flag for keys too
//                  large for them (formed once per source).
#include <algorithm>
#include <type_traits>

#include "internal.hpp"

namespace nmt {

// ----------------------------------------------------------- plain GEMM

// The row of a per-row table that batch row `row` reads: row itself without
// an index, else idx[row], or -1 where that is outside [0, nrows).
__device__ __forceinline__ int table_row(const int32_t* idx, int nrows, int row) {
  if (!idx) return row;
  const int r = idx[row];
  return r >= 0 && r < nrows ? r : -1;
}
// PlainEpi's added terms for output (row, n): add's gathered row, then add2's.
__device__ __forceinline__ float plain_add(const PlainEpi& ep, int row, int n) {
  float v = 0.f;
  if (ep.add) {
    const int r = table_row(ep.add_row, ep.add_rows, row);
    v = r >= 0 ? ep.add[(int64_t)r * ep.ld_add + n] : 0.f;
  }
  if (ep.add2) v += ep.add2[(int64_t)row * ep.ld_add2 + n];
  return v;
}

template <int TM, int TN, int WM, int WN, class P>
__global__ __launch_bounds__((TM / WM) * (TN / WN) * 64) void k_gemm_plain(AOperand A, const f32x4* __restrict__ Wp,
                                                                           int64_t Npad, PlainEpi ep) {
  constexpr int NT = (TM / WM) * (TN / WN) * 64;
  constexpr int FM = WM / 32, FN = WN / 32;
  __shared__ f32x4 lds[2 * (a_rows<TM, P>() + TN) * P::KQ];
  const int m0 = blockIdx.x * TM, n0 = blockIdx.y * TN;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wm0 = (wave % (TM / WM)) * WM, wn0 = (wave / (TM / WM)) * WN;
  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16{};

  int c_begin = 0, c_end = 1 << 30;
  if (ep.ksplit > 1) {
    const int nc = total_chunks(A);
    c_begin = (int)((int64_t)nc * blockIdx.z / ep.ksplit);
    c_end = (int)((int64_t)nc * (blockIdx.z + 1) / ep.ksplit);
  }
  // fp32: each k group's fragment reads go out during the previous group's
  // MFMAs (readout 72 -> 69.5 us, query 43 -> 41.5 us); bf16 (one MFMA per
  // k group and wave) keeps the compiler's order (readout 54 vs 56 us).
  using KS = std::conditional_t<P::kBF16, void, KgShape<FM + FN, 4 * FM * FN>>;
  gemm_mainloop<TM, TN, NT, P, kPlainLA<P>, KS>(
      A, Wp, Npad, m0, n0, lds,
      [&](const f32x4* As, const f32x4* Bs) {
#pragma unroll
        for (int kg = 0; kg < P::KQ / 2; ++kg) {
          f32x4 a[FM], b[FN];
#pragma unroll
          for (int i = 0; i < FM; ++i) a[i] = lds_frag_a<TM, P>(As, kg, wm0 + 32 * i);
#pragma unroll
          for (int j = 0; j < FN; ++j) b[j] = lds_frag<TN>(Bs, kg, wn0 + 32 * j);
#pragma unroll
          for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) P::mma(a[i], b[j], acc[i][j]);
        }
      },
      c_begin, c_end);

  const int h = lane >> 5, l32 = lane & 31;
  if (ep.ksplit > 1) {  // raw partial sums; k_splitk_reduce applies the epilogue
    float* part = ep.part + (int64_t)blockIdx.z * A.M * ep.N;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = n0 + wn0 + 32 * j + l32;
      if (n >= ep.N) continue;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + wm0 + 32 * i + acc_row(r, h);
          if (row < A.M) part[(int64_t)row * ep.N + n] = acc[i][j][r];
        }
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const int n = n0 + wn0 + 32 * j + l32;
    if (n >= ep.N) continue;
    const float bn = ep.bias ? ep.bias[n] : 0.f;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm0 + 32 * i + acc_row(r, h);
        if (row >= A.M) continue;
        float v = acc[i][j][r] + plain_add(ep, row, n) + bn;
        if (ep.act == 1) v = tanhf_(v);
        if (ep.mask_len && (row % ep.mask_T) >= ep.mask_len[row / ep.mask_T]) v = 0.f;
        if (ep.out16)
          ep.out16[(int64_t)row * ep.ldo + n] = (__bf16)v;
        else
          ep.out[(int64_t)row * ep.ldo + n] = v;
      }
  }
}

// Sums the split-K partials in split order, then bias, activation and mask.
__global__ void k_splitk_reduce(int M, int N, int ksplit, const float* __restrict__ part, PlainEpi ep) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)M * N) return;
  const int row = (int)(i / N), n = (int)(i % N);
  float v = 0.f;
  for (int z = 0; z < ksplit; ++z) v += part[(int64_t)z * M * N + i];
  v += plain_add(ep, row, n);
  v += ep.bias ? ep.bias[n] : 0.f;
  if (ep.act == 1) v = tanhf_(v);
  if (ep.mask_len && (row % ep.mask_T) >= ep.mask_len[row / ep.mask_T]) v = 0.f;
  if (ep.out16)
    ep.out16[(int64_t)row * ep.ldo + n] = (__bf16)v;
  else
    ep.out[(int64_t)row * ep.ldo + n] = v;
}

// The same for four consecutive columns per thread (N, the row strides and
// the arrays' alignment allowing 16-byte accesses).
__global__ void k_splitk_reduce4(int M, int N, int ksplit, const float* __restrict__ part, PlainEpi ep) {
  const int64_t i4 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x, n4 = N / 4;
  if (i4 >= (int64_t)M * n4) return;
  const int row = (int)(i4 / n4), n = 4 * (int)(i4 % n4);
  const int64_t i = (int64_t)row * N + n;
  f32x4 v = zero4();
  for (int z = 0; z < ksplit; ++z) v += *(const f32x4*)(part + (int64_t)z * M * N + i);
  f32x4 t = zero4();  // the added terms, summed as plain_add sums them
  if (ep.add) {
    const int r = table_row(ep.add_row, ep.add_rows, row);
    if (r >= 0) t = *(const f32x4*)(ep.add + (int64_t)r * ep.ld_add + n);
  }
  if (ep.add2) t += *(const f32x4*)(ep.add2 + (int64_t)row * ep.ld_add2 + n);
  v += t;
  if (ep.bias) v += *(const f32x4*)(ep.bias + n);
  const bool masked = ep.mask_len && (row % ep.mask_T) >= ep.mask_len[row / ep.mask_T];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if (ep.act == 1) v[e] = tanhf_(v[e]);
    if (masked) v[e] = 0.f;
  }
  if (ep.out16) {
    typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
    *(bf16x4_t*)(ep.out16 + (int64_t)row * ep.ldo + n) = bf16x4_t{(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
  } else {
    *(f32x4*)(ep.out + (int64_t)row * ep.ldo + n) = v;
  }
}

static bool reduce4_fits(const PlainEpi& ep, const float* part) {
  auto al = [](const void* p, int b) { return ((uintptr_t)p % b) == 0; };
  return ep.N % 4 == 0 && ep.ldo % 4 == 0 && al(part, 16) && (ep.out16 ? al(ep.out16, 8) : al(ep.out, 16)) &&
         (!ep.bias || al(ep.bias, 16)) && (!ep.add || (ep.ld_add % 4 == 0 && al(ep.add, 16))) &&
         (!ep.add2 || (ep.ld_add2 % 4 == 0 && al(ep.add2, 16)));
}

template <int TM, int TN, int WM, int WN, class P>
static void plain_tile(const AOperand& A, const f32x4* Wp, const Packed& W, const PlainEpi& ep, int ksplit,
                       hipStream_t st) {
  dim3 grid(ceil_div(A.M, TM), (unsigned)(W.Npad / TN), ksplit);
  hipLaunchKernelGGL((k_gemm_plain<TM, TN, WM, WN, P>), grid, dim3((TM / WM) * (TN / WN) * 64), 0, st, A, Wp,
                     W.Npad, ep);
}

template <class P>
hipError_t gemm_plain(Tile t, const AOperand& A, const Packed& W, const PlainEpi& ep, hipStream_t st) {
  const f32x4* Wp = (const f32x4*)W.d;
  if (W.Npad % tile_n(t)) return hipErrorInvalidValue;
  if (ep.ksplit > 1 && !ep.part) return hipErrorInvalidValue;
  const int ks = ep.ksplit > 1 ? ep.ksplit : 1;
  if (t == Tile::Small)
    plain_tile<kPlainSmallTM, kPlainSmallTN, 32, 32, P>(A, Wp, W, ep, ks, st);
  else
    plain_tile<kPlainLargeTM, kPlainLargeTN, 64, 64, P>(A, Wp, W, ep, ks, st);
  if (ep.ksplit > 1 && !ep.defer_reduce) {
    const int64_t n = (int64_t)A.M * ep.N;
    if (reduce4_fits(ep, ep.part))
      hipLaunchKernelGGL(k_splitk_reduce4, dim3(ceil_div(n / 4, 256)), dim3(256), 0, st, A.M, ep.N, ep.ksplit, ep.part,
                         ep);
    else
      hipLaunchKernelGGL(k_splitk_reduce, dim3(ceil_div(n, 256)), dim3(256), 0, st, A.M, ep.N, ep.ksplit, ep.part, ep);
  }
  return hipGetLastError();
}

// Each segment with work needs a matrix behind it, and the staging
// addresses the segments and the packed weights with 32-bit byte offsets.
static bool segments_loadable(const AOperand& A, int64_t Npad, bool bf16) {
  int64_t chunks = 0;
  for (int i = 0; i < A.nseg; ++i) {
    const ASeg& s = A.seg[i];
    if (s.nchunk <= 0) continue;
    if (!s.p || (s.gather && s.gmax < 1)) return false;
    if ((int64_t)(s.gather ? s.gmax : A.M) * s.ld * (s.bf16 ? 2 : 4) >= ((int64_t)1 << 31)) return false;
    chunks += s.nchunk;
  }
  return chunks * (bf16 ? PrecBF16::KQ : PrecF32::KQ) * Npad * 16 < ((int64_t)1 << 31);
}

static bool try_plain_ws(const AOperand& A, const Packed& W, const PlainEpi& ep, int cus, hipStream_t st);

hipError_t launch_gemm_plain(Tile t, const AOperand& A, const Packed& W, const PlainEpi& ep, hipStream_t st,
                             int cus) {
  if (A.M <= 0 || ep.N <= 0) return hipSuccess;
  if (!segments_loadable(A, W.Npad, W.bf16)) return hipErrorInvalidValue;
  if (t == Tile::Small && try_plain_ws(A, W, ep, cus, st)) return hipGetLastError();
  return W.bf16 ? gemm_plain<PrecBF16>(t, A, W, ep, st) : gemm_plain<PrecF32>(t, A, W, ep, st);
}

// ------------------------------------------------------------- GRU GEMM

struct GruBatch {
  GruProblem p[2];
  int32_t ksplit;  // SPLIT kernels: K splits per problem (blockIdx.z = problem * ksplit + split)
  float* part;     // SPLIT kernels: raw sums [problem][split][M][4][H] (r, z, input and state candidate)
  int32_t part_M;  // rows of each problem's part block
};

// The cell of Section 5.1's GRUs from the gate pre-activations (without
// biases) and the previous state.
__device__ __forceinline__ float gru_cell(float sr, float sz, float sni, float sns, float br, float bz, float bni,
                                          float bns, float xr, float xz, float xn, float hp) {
  const float rg = sigmoidf_(sr + br + xr);
  const float zg = sigmoidf_(sz + bz + xz);
  const float ng = tanhf_(sni + bni + xn + rg * (sns + bns));
  return zg * hp + (1.f - zg) * ng;
}

// SPLIT: the block sums only its split's share of the K chunks (of all A
// segments together) and writes the raw sums to batch.part; k_gru_cell adds
// the splits in order and applies the cell.  For launches with few row
// tiles (the encoder's recurrence over S rows), which would otherwise leave
// most CUs idle.
template <int TM, int HB, int WM, class P, bool SPLIT = false>
__global__ __launch_bounds__((TM / WM) * (HB / 32) * 64) __attribute__((amdgpu_waves_per_eu(2))) void k_gemm_gru(
    GruBatch batch) {
  constexpr int TN = 3 * HB;
  constexpr int NT = (TM / WM) * (HB / 32) * 64;
  constexpr int FM = WM / 32;
  __shared__ f32x4 lds[2 * (a_rows<TM, P>() + TN) * P::KQ];
  const int prob = SPLIT ? (int)blockIdx.z / batch.ksplit : (int)blockIdx.z;
  const int split = SPLIT ? (int)blockIdx.z % batch.ksplit : 0;
  const GruProblem& Pb = batch.p[prob];
  const f32x4* Wp = (const f32x4*)Pb.Wp;
  const int m0 = blockIdx.x * TM, n0 = blockIdx.y * TN;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wm0 = (wave % (TM / WM)) * WM, wu0 = (wave / (TM / WM)) * 32;
  f32x16 ar[FM], az[FM], ani[FM], ans[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) ar[i] = az[i] = ani[i] = ans[i] = f32x16{};
  auto chunk = [&](const f32x4* As, const f32x4* Bs, auto state_side) {
#pragma unroll
    for (int kg = 0; kg < P::KQ / 2; ++kg) {
      f32x4 a[FM];
#pragma unroll
      for (int i = 0; i < FM; ++i) a[i] = lds_frag_a<TM, P>(As, kg, wm0 + 32 * i);
      const f32x4 br = lds_frag<TN>(Bs, kg, wu0);
      const f32x4 bz = lds_frag<TN>(Bs, kg, HB + wu0);
      const f32x4 bn = lds_frag<TN>(Bs, kg, 2 * HB + wu0);
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        P::mma(a[i], br, ar[i]);
        P::mma(a[i], bz, az[i]);
        if constexpr (decltype(state_side)::value)
          P::mma(a[i], bn, ans[i]);
        else
          P::mma(a[i], bn, ani[i]);
      }
    }
  };
  // bf16: each k group's fragment reads go out during the previous group's
  // MFMAs (GRU2 116 -> 112 us); fp32 (12 MFMAs per k group) keeps the
  // compiler's order, which measured faster there (287 vs 295 us).
  using KS = std::conditional_t<P::kBF16, KgShape<FM + 3, 3 * FM>, void>;
  // One main loop per A segment, each with its side fixed at compile time:
  // a per-chunk branch between the two candidate accumulators would make the
  // compiler shuttle every accumulator between AGPRs and VGPRs each chunk.
  // this block's global chunk range (all of them without a split)
  int c_begin = 0, c_end = 1 << 30;
  if constexpr (SPLIT) {
    const int nc = total_chunks(Pb.A);
    c_begin = (int)((int64_t)nc * split / batch.ksplit);
    c_end = (int)((int64_t)nc * (split + 1) / batch.ksplit);
  }
  int64_t vq0 = 0;
  int s0 = 0;
  for (int sg = 0; sg < Pb.A.nseg; ++sg) {
    const ASeg seg = seg_at(Pb.A, sg);
    const int cb = c_begin > s0 ? c_begin - s0 : 0;
    const int ce = c_end - s0 < seg.nchunk ? c_end - s0 : seg.nchunk;
    if (seg.side)
      gemm_segment<TM, TN, NT, P, kGruLA<P>, KS>(
          seg, Pb.A.M, Wp, Pb.Npad, m0, n0, lds,
          [&](const f32x4* As, const f32x4* Bs) { chunk(As, Bs, std::true_type{}); }, vq0, cb, ce);
    else
      gemm_segment<TM, TN, NT, P, kGruLA<P>, KS>(
          seg, Pb.A.M, Wp, Pb.Npad, m0, n0, lds,
          [&](const f32x4* As, const f32x4* Bs) { chunk(As, Bs, std::false_type{}); }, vq0, cb, ce);
    vq0 += (int64_t)seg.nchunk * P::KQ;
    s0 += seg.nchunk;
  }

  const GruEpi& ep = Pb.ep;
  const int h = lane >> 5, l32 = lane & 31;
  const int H = ep.H, M = Pb.A.M;
  const int j = blockIdx.y * HB + wu0 + l32;
  if (j >= H) return;
  if constexpr (SPLIT) {
    float* part = batch.part + ((int64_t)prob * batch.ksplit + split) * batch.part_M * 4 * H;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm0 + 32 * i + acc_row(r, h);
        if (row >= M) continue;
        float* o = part + (int64_t)row * 4 * H + j;
        o[0] = ar[i][r];
        o[H] = az[i][r];
        o[2 * H] = ani[i][r];
        o[3 * H] = ans[i][r];
      }
    return;
  }
  const float br = ep.brz[j], bz = ep.brz[H + j], bni = ep.bni[j], bns = ep.bns[j];
  // The cell's other inputs for this lane's rows, 8 rows at a time, every
  // load of a group issued before any value is used (addresses clamped to
  // row 0 where a row is absent), so the epilogue waits for memory a few
  // times per group instead of once per row.
  constexpr int NG = 8;
  auto clamp_row = [&](int row) { return row < M ? row : 0; };
#pragma unroll
  for (int g0 = 0; g0 < FM * 16; g0 += NG) {
    int rowq[NG];
    float hp[NG], xr[NG], xz[NG], xn[NG];
    bool keep[NG];
#pragma unroll
    for (int q = 0; q < NG; ++q) {
      rowq[q] = m0 + wm0 + 32 * ((g0 + q) / 16) + acc_row((g0 + q) % 16, h);
      hp[q] = xr[q] = xz[q] = xn[q] = 0.f;
      keep[q] = true;
    }
    if (ep.h) {
      int hr[NG];
      bool hok[NG];
#pragma unroll
      for (int q = 0; q < NG; ++q) hr[q] = ep.hrow ? ep.hrow[clamp_row(rowq[q])] : clamp_row(rowq[q]);
#pragma unroll
      for (int q = 0; q < NG; ++q) {
        hok[q] = !ep.hrow || (hr[q] >= 0 && hr[q] < ep.hrows);
        hp[q] = ep.h[(int64_t)(hok[q] ? hr[q] : 0) * ep.ldh + j];
      }
#pragma unroll
      for (int q = 0; q < NG; ++q) hp[q] = hok[q] ? hp[q] : 0.f;
    }
    if (ep.xin) {
      int xq[NG];
#pragma unroll
      for (int q = 0; q < NG; ++q) xq[q] = table_row(ep.xrow, ep.xrows, clamp_row(rowq[q]));
#pragma unroll
      for (int q = 0; q < NG; ++q) {
        const float* x = ep.xin + (int64_t)(xq[q] >= 0 ? xq[q] : 0) * ep.ldx;
        xr[q] = x[j];
        xz[q] = x[H + j];
        xn[q] = x[2 * H + j];
      }
#pragma unroll
      for (int q = 0; q < NG; ++q)
        if (xq[q] < 0) xr[q] = xz[q] = xn[q] = 0.f;
    }
    if (ep.mask_len) {
#pragma unroll
      for (int q = 0; q < NG; ++q) keep[q] = ep.mask_pos < ep.mask_len[clamp_row(rowq[q])];
    }
#pragma unroll
    for (int q = 0; q < NG; ++q) {
      const int i = (g0 + q) / 16, r = (g0 + q) % 16;
      float hn = gru_cell(ar[i][r], az[i][r], ani[i][r], ans[i][r], br, bz, bni, bns, xr[q], xz[q], xn[q], hp[q]);
      if (!keep[q]) hn = 0.f;
      if (rowq[q] < M) {
        ep.out[(int64_t)rowq[q] * ep.ldo + j] = hn;
        if (ep.out16) ep.out16[(int64_t)rowq[q] * ep.ldo + j] = (__bf16)hn;
      }
    }
  }
}

static bool try_gru_ws(const GruProblem& p, int H, bool bf16, int cus, hipStream_t st);

hipError_t launch_gemm_gru(const GruProblem* probs, int nprob, int H, bool bf16, int cus, hipStream_t st) {
  if (nprob < 1 || nprob > 2) return hipErrorInvalidValue;
  GruBatch b{};
  b.p[0] = probs[0];
  b.p[1] = nprob > 1 ? probs[1] : probs[0];
  int M = probs[0].A.M;
  for (int i = 1; i < nprob; ++i) M = M > probs[i].A.M ? M : probs[i].A.M;
  if (M <= 0) return hipSuccess;
  for (int i = 0; i < nprob; ++i)
    if (!segments_loadable(probs[i].A, probs[i].Npad, bf16)) return hipErrorInvalidValue;
  // Batches too small to give every CU a block of the large tile (a forest
  // level of about 1,000 rows, the encoder's recurrence) take blocks of
  // kGruSmallTM rows instead, twice as many, which run two to a CU.
  auto run = [&](auto tm, auto hb, auto wm, auto prec) {
    constexpr int TM = decltype(tm)::value, HB = decltype(hb)::value, WM = decltype(wm)::value;
    using P = decltype(prec);
    dim3 grid(ceil_div(M, TM), ceil_div(H, HB), nprob);
    hipLaunchKernelGGL((k_gemm_gru<TM, HB, WM, P>), grid, dim3((TM / WM) * (HB / 32) * 64), 0, st, b);
  };
  if (nprob == 1 && try_gru_ws(probs[0], H, bf16, cus, st)) return hipGetLastError();
  const int tm_large = bf16 ? kGruTM16 : kGruTM, hb = gru_hb(bf16);
  // fp32 also when the large tile's last round would be at most half full
  // (B = 2500 and 3000: GRU2 544 -> 434-440 us); bf16 there measured slower.
  const int64_t nbl = (int64_t)ceil_div(M, tm_large) * ceil_div(H, hb) * nprob;
  const int64_t last = nbl % cus;
  const bool small = nbl < cus || (!bf16 && last != 0 && last <= cus / 2);
  if (bf16) {
    if (small)
      run(std::integral_constant<int, kGruSmallTM>{}, std::integral_constant<int, kGruHB16>{},
          std::integral_constant<int, kGruWM16>{}, PrecBF16{});
    else
      run(std::integral_constant<int, kGruTM16>{}, std::integral_constant<int, kGruHB16>{},
          std::integral_constant<int, kGruWM16>{}, PrecBF16{});
  } else {
    if (small)
      run(std::integral_constant<int, kGruSmallTM>{}, std::integral_constant<int, kGruHB>{},
          std::integral_constant<int, kGruWM>{}, PrecF32{});
    else
      run(std::integral_constant<int, kGruTM>{}, std::integral_constant<int, kGruHB>{},
          std::integral_constant<int, kGruWM>{}, PrecF32{});
  }
  return hipGetLastError();
}

int gru_split_tm(int M, int H, bool bf16, int cus) {
  return 2 * (int64_t)ceil_div(M, kGruTM) * ceil_div(H, gru_hb(bf16)) >= cus ? kGruTM : kGruSmallTM;
}

int gru_ksplit(int M, int H, int nchunks, bool bf16, int cus) {
  const int tm = gru_split_tm(M, H, bf16, cus);
  const int64_t blocks = (int64_t)ceil_div(M, tm) * ceil_div(H, gru_hb(bf16));
  // about two 4-wave blocks per CU, or one 8-wave block
  const int64_t target = tm == kGruSmallTM ? 2 * (int64_t)cus : (int64_t)cus;
  int ks = (int)std::min<int64_t>(8, target / std::max<int64_t>(blocks, 1));
  ks = std::min(ks, nchunks / 4);
  return ks < 2 ? 1 : ks;
}

// Adds the K splits of a SPLIT launch in split order and applies the cell,
// with the same inputs and outputs as the fused epilogue.  One thread per
// (row, hidden unit) of problem blockIdx.y.
__global__ void k_gru_cell(GruBatch batch, int H) {
  const GruProblem& Pb = batch.p[blockIdx.y];
  const GruEpi& ep = Pb.ep;
  const int M = Pb.A.M;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)M * H) return;
  const int row = (int)(i / H), j = (int)(i % H);
  const int64_t stride = (int64_t)batch.part_M * 4 * H;
  const float* p = batch.part + (int64_t)blockIdx.y * batch.ksplit * stride + (int64_t)row * 4 * H + j;
  float sr = 0.f, sz = 0.f, sni = 0.f, sns = 0.f;
  for (int z = 0; z < batch.ksplit; ++z, p += stride) {
    sr += p[0];
    sz += p[H];
    sni += p[2 * H];
    sns += p[3 * H];
  }
  float hp = 0.f, xr = 0.f, xz = 0.f, xn = 0.f;
  if (ep.h) {
    const int hr = ep.hrow ? ep.hrow[row] : row;
    if (!ep.hrow || (hr >= 0 && hr < ep.hrows)) hp = ep.h[(int64_t)hr * ep.ldh + j];
  }
  const int xq = ep.xin ? table_row(ep.xrow, ep.xrows, row) : -1;
  if (xq >= 0) {
    const float* x = ep.xin + (int64_t)xq * ep.ldx;
    xr = x[j];
    xz = x[H + j];
    xn = x[2 * H + j];
  }
  float hn = gru_cell(sr, sz, sni, sns, ep.brz[j], ep.brz[H + j], ep.bni[j], ep.bns[j], xr, xz, xn, hp);
  if (ep.mask_len && ep.mask_pos >= ep.mask_len[row]) hn = 0.f;
  ep.out[(int64_t)row * ep.ldo + j] = hn;
  if (ep.out16) ep.out16[(int64_t)row * ep.ldo + j] = (__bf16)hn;
}

hipError_t launch_gemm_gru_split(const GruProblem* probs, int nprob, int H, bool bf16, int ksplit, float* part,
                                 int part_M, int tm, hipStream_t st) {
  if (nprob < 1 || nprob > 2 || ksplit < 1 || !part) return hipErrorInvalidValue;
  GruBatch b{};
  b.p[0] = probs[0];
  b.p[1] = nprob > 1 ? probs[1] : probs[0];
  b.ksplit = ksplit;
  b.part = part;
  b.part_M = part_M;
  int M = 0;
  for (int i = 0; i < nprob; ++i) {
    if (probs[i].A.M > part_M) return hipErrorInvalidValue;
    if (!segments_loadable(probs[i].A, probs[i].Npad, bf16)) return hipErrorInvalidValue;
    M = M > probs[i].A.M ? M : probs[i].A.M;
  }
  if (M <= 0) return hipSuccess;
  if (tm != kGruSmallTM && tm != kGruTM) return hipErrorInvalidValue;
  auto run = [&](auto tmc) {
    constexpr int TM = decltype(tmc)::value;
    if (bf16)
      hipLaunchKernelGGL((k_gemm_gru<TM, kGruHB16, kGruWM16, PrecBF16, true>),
                         dim3(ceil_div(M, TM), ceil_div(H, kGruHB16), nprob * ksplit),
                         dim3((TM / kGruWM16) * (kGruHB16 / 32) * 64), 0, st, b);
    else
      hipLaunchKernelGGL((k_gemm_gru<TM, kGruHB, kGruWM, PrecF32, true>),
                         dim3(ceil_div(M, TM), ceil_div(H, kGruHB), nprob * ksplit),
                         dim3((TM / kGruWM) * (kGruHB / 32) * 64), 0, st, b);
  };
  if (tm == kGruTM)
    run(std::integral_constant<int, kGruTM>{});
  else
    run(std::integral_constant<int, kGruSmallTM>{});
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_gru_cell, dim3(ceil_div((int64_t)M * H, (int64_t)256), nprob), dim3(256), 0, st, b, H);
  return hipGetLastError();
}

// ------------------------------------- weight-streaming GRU GEMM (bf16 weights)
//
// With bf16 weights the LDS-staged GRU tile above runs MFMAs 8x faster per k
// than with fp32 ones, so the fixed costs of each 64-k chunk (the staging
// loads, the transposed LDS stores of both operands, the barrier) dominate
// it (GRU2 at B = 4096: 38 % MFMA busy).  This form keeps only the
// activations in LDS and streams the packed weights from L2 straight into
// registers, as the vocabulary kernel does.  A block holds 128 rows x 128
// hidden units; wave w computes rows 64 (w & 1) .. 64 (w & 1) + 63 and units
// 32 (w >> 1) .. of the block, all three gates with the candidate split by
// side, so each weight fragment feeds two MFMAs and each activation fragment
// three.  Activations go through registers into one of two LDS stages in
// chunks of 128 k, one barrier per 8 k steps.  The MFMA puts the weights on
// its row operand and the activations on its column operand, so register r of
// a lane's gate accumulator is unit 8 (r / 4) + 4 h + r % 4 of the wave's 32
// for the lane's batch row: the cell runs lane-locally in the epilogue.
// Used for an A operand of two segments in whole 128-k chunks, one on each
// side: FIRST_STATE says whether segment 0 is the state side (the second
// GRU: [s1 | c]) or the input side (the first: [x | s_prev]), SRC16_i
// whether segment i is stored in bf16 (else fp32, rounded to bf16 as it is
// staged; its second staging register set leaves room for 2 weight steps in
// flight, which measured the same as 4).  Taken when the grid covers the CUs.
constexpr int kWsTM = 128, kWsUB = 128, kWsKQ = 16;
#ifndef NMT_WS_VPF_BF16_SRC   // weight steps in flight, both segments bf16
#define NMT_WS_VPF_BF16_SRC 4
#endif
#ifndef NMT_WS_VPF_F32_SRC    // weight steps in flight with an fp32 segment
#define NMT_WS_VPF_F32_SRC 2
#endif

template <bool FIRST_STATE, bool SRC16_0, bool SRC16_1, int VPF>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2))) void k_gru_ws(GruProblem Pb) {
  using P = PrecBF16;
  constexpr int TM = kWsTM, KQW = kWsKQ, NKS = KQW / 2, NT = 512;
  constexpr int NA = TM * KQW / NT;  // activation vectors per thread per chunk
  static_assert(NKS % VPF == 0, "ring slots fixed within a chunk");
  __shared__ f32x4 As[2 * KQW * TM];  // [stage][vector][row ^ (vector & 15)]
  const AOperand& A = Pb.A;
  const int M = A.M;
  const int m0 = blockIdx.x * TM;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int h = lane >> 5, l32 = lane & 31, wr = wave & 1;
  const int u0 = blockIdx.y * kWsUB + 32 * (wave >> 1);
  const int64_t Npad = Pb.Npad;
  const int nch = total_chunks(A) / 2;  // 128-k chunks
  const int last_gk = nch * NKS - 1;
  // weights: packed column tile u0 / HB holds [r | z | n] of HB units, and a
  // wave's 32 units lie in one tile
  constexpr int HB = kGruHB16;
  static_assert(HB % 32 == 0, "a wave's units within one packed tile");
  const int c_r = (u0 / HB) * 3 * HB + u0 % HB;
  const __amdgpu_buffer_rsrc_t wres = buffer_rsrc(Pb.Wp, (int64_t)nch * KQW * Npad * 16);
  const int lo_r = (int)(((int64_t)h * Npad + c_r + l32) * 16);
  const int lo_z = lo_r + HB * 16, lo_n = lo_r + 2 * HB * 16;
  const int kbytes = (int)(2 * Npad * 16);  // one k step: two packed vector rows
  auto wload = [&](f32x4(&d)[3], int gk) {
    const int so = (gk < last_gk ? gk : last_gk) * kbytes;  // past the end: re-read the last step (unused)
    d[0] = buf_load(wres, lo_r, so);
    d[1] = buf_load(wres, lo_z, so);
    d[2] = buf_load(wres, lo_n, so);
  };

  // activation staging: this thread's vectors are rows tid / KQW + 32 i,
  // vector tid % KQW of each chunk, from segment 0 (the first c1 chunks) or
  // segment 1
  static_assert(NT / KQW == 32 && KQW == 16, "staging rows 32 apart");
  const ASeg sg0 = seg_at(A, 0), sg1 = seg_at(A, 1);
  const int c1 = sg0.nchunk / 2;
  const __amdgpu_buffer_rsrc_t res0 = buffer_rsrc(sg0.p, seg_bytes(sg0, M));
  const __amdgpu_buffer_rsrc_t res1 = buffer_rsrc(sg1.p, seg_bytes(sg1, M));
  const int kin = P::KV * ((int)threadIdx.x % KQW);
  int roff0[NA], roff1[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int row = m0 + ((int)threadIdx.x + i * NT) / KQW;
    roff0[i] = seg_row_off(sg0, row, M);
    roff1[i] = seg_row_off(sg1, row, M);
  }
  f32x4 ra[NA], rb[NA];  // rb: the second half of an fp32 source vector
  auto aload = [&](int c) {  // chunk c of the whole A
    if constexpr (SRC16_0 == SRC16_1) {
      // one load sequence with the segment's resource, offsets and width
      // selected (a branch here gets merged by the compiler into a
      // dynamically indexed copy of the segments in scratch memory)
      const bool second = c >= c1;
      const int kseg = (second ? c - c1 : c) * KQW * P::KV;
      const int K = second ? sg1.K : sg0.K;
#pragma unroll
      for (int i = 0; i < NA; ++i)
        load_a_raw<P, SRC16_0>(second ? res1 : res0, second ? roff1[i] : roff0[i], K, kseg + kin, kin,
                               kseg * (SRC16_0 ? 2 : 4), ra[i], rb[i]);
    } else if (c < c1) {  // a uniform branch between the two load sequences
      const int kseg = c * KQW * P::KV;
#pragma unroll
      for (int i = 0; i < NA; ++i)
        load_a_raw<P, SRC16_0>(res0, roff0[i], sg0.K, kseg + kin, kin, kseg * (SRC16_0 ? 2 : 4), ra[i], rb[i]);
    } else {
      const int kseg = (c - c1) * KQW * P::KV;
#pragma unroll
      for (int i = 0; i < NA; ++i)
        load_a_raw<P, SRC16_1>(res1, roff1[i], sg1.K, kseg + kin, kin, kseg * (SRC16_1 ? 2 : 4), ra[i], rb[i]);
    }
  };
  // (row ^ v) = (tid / KQW ^ v) + 32 i for row = tid / KQW + 32 i and v < 16:
  // one swizzled base per thread, the rest immediate offsets
  const int st_base = ((int)threadIdx.x % KQW) * TM + (((int)threadIdx.x / KQW) ^ ((int)threadIdx.x % KQW));
  auto astore = [&](int stage, int c) {  // c: the chunk the staged data belongs to
    const bool s16 = c < c1 ? SRC16_0 : SRC16_1;
#pragma unroll
    for (int i = 0; i < NA; ++i)
      As[stage * KQW * TM + st_base + 32 * i] = s16 ? ra[i] : a_from_raw<P, false>(ra[i], rb[i]);
  };
  // fragment of k step ks (vectors 2 ks + h) for the 32 rows at r0;
  // (r0 + l32) ^ v = r0 + (l32 ^ v) for r0 a multiple of 32 and v < 16
  auto afrag = [&](int stage, int ks, int r0) {
    const int v = 2 * ks + h;
    return As[stage * KQW * TM + r0 + v * TM + (l32 ^ v)];
  };

  f32x16 ar[2], az[2], ani[2], ans[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) ar[i] = az[i] = ani[i] = ans[i] = f32x16{};
  f32x4 ring[VPF][3];
#pragma unroll
  for (int p = 0; p < VPF; ++p) wload(ring[p], p);
  aload(0);
  astore(0, 0);
  if (nch > 1) aload(1);
  __syncthreads();

  const int r0 = 64 * wr;
  // Chunks [cb, ce) of one segment, its side fixed at compile time (a
  // per-chunk branch would shuttle the accumulators between register files).
  auto run = [&](int cb, int ce, auto side_c) {
    constexpr bool SIDE = decltype(side_c)::value;
    for (int c = cb; c < ce; ++c) {
      const int st = c & 1;
      f32x4 a0 = afrag(st, 0, r0), a1 = afrag(st, 0, r0 + 32);
      static_for<NKS>([&](auto kc) {
        constexpr int ks = decltype(kc)::value, slot = ks % VPF;
        f32x4 n0 = a0, n1 = a1;
        if constexpr (ks + 1 < NKS) {
          n0 = afrag(st, ks + 1, r0);
          n1 = afrag(st, ks + 1, r0 + 32);
        }
        P::mma(ring[slot][0], a0, ar[0]);
        P::mma(ring[slot][0], a1, ar[1]);
        P::mma(ring[slot][1], a0, az[0]);
        P::mma(ring[slot][1], a1, az[1]);
        if constexpr (SIDE) {
          P::mma(ring[slot][2], a0, ans[0]);
          P::mma(ring[slot][2], a1, ans[1]);
        } else {
          P::mma(ring[slot][2], a0, ani[0]);
          P::mma(ring[slot][2], a1, ani[1]);
        }
        wload(ring[slot], c * NKS + ks + VPF);  // refill the slot just consumed, VPF steps ahead
        // one MFMA, the next step's fragment reads, the other MFMAs, the refill
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 5, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 3, 0);
        a0 = n0;
        a1 = n1;
      });
      if (c + 1 < nch) astore(st ^ 1, c + 1);
      if (c + 2 < nch) aload(c + 2);
      __syncthreads();
    }
  };
  // segment 0's side, then segment 1's (each fixed at compile time; a runtime
  // choice between the two loops doubled the live registers)
  run(0, c1, std::integral_constant<bool, FIRST_STATE>{});
  run(c1, nch, std::integral_constant<bool, !FIRST_STATE>{});

  // the cell, lane-locally: register r of row fragment i is unit u0 + 8 (r / 4) + 4 h + r % 4 of row r0 + 32 i + l32
  const GruEpi& ep = Pb.ep;
  const int H = ep.H;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int row = m0 + r0 + 32 * i + l32;
    if (row >= M) continue;
    int hr = row;
    bool hok = true;
    if (ep.h && ep.hrow) {
      hr = ep.hrow[row];
      hok = hr >= 0 && hr < ep.hrows;
    }
    const bool keep = !ep.mask_len || ep.mask_pos < ep.mask_len[row];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j0 = u0 + 8 * q + 4 * h;
      if (j0 >= H) continue;
      const f32x4 br = *(const f32x4*)(ep.brz + j0), bz = *(const f32x4*)(ep.brz + H + j0);
      const f32x4 bni = *(const f32x4*)(ep.bni + j0), bns = *(const f32x4*)(ep.bns + j0);
      const f32x4 hp = (ep.h && hok) ? *(const f32x4*)(ep.h + (int64_t)hr * ep.ldh + j0) : zero4();
      f32x4 xr = zero4(), xz = zero4(), xn = zero4();
      if (ep.xin) {
        const float* x = ep.xin + (int64_t)row * ep.ldx;
        xr = *(const f32x4*)(x + j0);
        xz = *(const f32x4*)(x + H + j0);
        xn = *(const f32x4*)(x + 2 * H + j0);
      }
      f32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 4 * q + e;
        const float hn = gru_cell(ar[i][r], az[i][r], ani[i][r], ans[i][r], br[e], bz[e], bni[e], bns[e], xr[e],
                                  xz[e], xn[e], hp[e]);
        o[e] = keep ? hn : 0.f;
      }
      *(f32x4*)(ep.out + (int64_t)row * ep.ldo + j0) = o;
      if (ep.out16) {
        typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
        *(bf16x4_t*)(ep.out16 + (int64_t)row * ep.ldo + j0) = bf16x4_t{(__bf16)o[0], (__bf16)o[1], (__bf16)o[2],
                                                                         (__bf16)o[3]};
      }
    }
  }
}

std::atomic<int> g_gemm_form{0};
std::atomic<int64_t> g_gemm_streamed{0};

static bool aligned(const void* p, int bytes) { return ((uintptr_t)p % bytes) == 0; }

// The weight-streaming form for one bf16 problem, if it applies (see above);
// returns false to let the caller launch the LDS-staged tile instead.
static bool try_gru_ws(const GruProblem& p, int H, bool bf16, int cus, hipStream_t st) {
  const int form = g_gemm_form.load(std::memory_order_relaxed);
  if (form == 2) return false;
  // H a multiple of the block's 128 units: every wave's packed columns then
  // lie inside the matrix's rows, so no weight load leaves the matrix
  if (!bf16 || H % kWsUB || p.A.M <= 0 || p.A.nseg != 2 || p.ep.xrow) return false;
  const ASeg &s0 = p.A.seg[0], &s1 = p.A.seg[1];
  if (s0.nchunk % 2 || s1.nchunk % 2 || s0.side == s1.side) return false;
  // the epilogue's vector accesses: 16-byte aligned rows of the state,
  // candidate input, output and bias arrays, 8-byte ones of the bf16 output
  const GruEpi& ep = p.ep;
  if ((ep.h && (ep.ldh % 4 || !aligned(ep.h, 16))) || ep.ldo % 4 || !aligned(ep.out, 16) ||
      (ep.out16 && !aligned(ep.out16, 8)) || (ep.xin && (ep.ldx % 4 || !aligned(ep.xin, 16))) ||
      !aligned(ep.brz, 16) || !aligned(ep.bni, 16) || !aligned(ep.bns, 16))
    return false;
  const int64_t blocks = (int64_t)ceil_div(p.A.M, kWsTM) * ceil_div(H, kWsUB);
  if (form == 0 && blocks < cus) return false;
  const dim3 grid(ceil_div(p.A.M, kWsTM), H / kWsUB), block(512);
  if (s0.side == 1 && s0.bf16 && s1.bf16)  // the second GRU: [s1 | c]
    hipLaunchKernelGGL((k_gru_ws<true, true, true, NMT_WS_VPF_BF16_SRC>), grid, block, 0, st, p);
  else if (s0.side == 0 && s0.bf16 && !s1.bf16)  // the first: [x | s_prev (fp32)]
    hipLaunchKernelGGL((k_gru_ws<false, true, false, NMT_WS_VPF_F32_SRC>), grid, block, 0, st, p);
  else
    return false;
  g_gemm_streamed.fetch_add(1, std::memory_order_relaxed);
  return true;
}

// ---------------------------------- weight-streaming plain GEMM (bf16 weights)
//
// The bf16 query and readout products in the form of k_gru_ws: activations
// staged through registers into LDS in 128-k chunks, packed weights streamed
// from L2 straight into registers.  A wave computes 64 rows x 32 columns
// (each weight fragment feeds two MFMAs); a block of 8 waves covers 128 rows
// and 128 columns (KSPLIT = 1), or 64 columns with the 8 k steps of each
// chunk shared between two groups of four waves (KSPLIT = 2, where 128-column
// blocks would leave CUs idle: the readout's 512 columns), whose sums meet in
// LDS before the epilogue.  Segment 0 of A may be fp32 (rounded to bf16 as it
// is staged); the others are bf16.  The output layout matches the GRU form:
// register r of row fragment i is column 8 (r / 4) + 4 h + r % 4 of the
// wave's 32 for batch row 32 i + l32, so a lane stores 4 consecutive columns.
#ifndef NMT_PW_VPF  // weight steps in flight
#define NMT_PW_VPF 4
#endif
constexpr int kPwTM = 128, kPwKQ = 16, kPwVPF = NMT_PW_VPF;

template <int NSEG, bool SRC16_0, int KSPLIT>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2))) void k_plain_ws(AOperand A, const void* Wp,
                                                                                         int64_t Npad, PlainEpi ep) {
  using P = PrecBF16;
  constexpr int TM = kPwTM, KQW = kPwKQ, NKS = KQW / 2, NT = 512;
  constexpr int NA = TM * KQW / NT;  // activation vectors per thread per chunk
  constexpr int NKL = NKS / KSPLIT;  // k steps per chunk and wave
  // Activation chunks in flight in registers: the readout (three segments,
  // one of them fp32) alternates two register sets, so a chunk's loads have
  // two chunks' MFMAs to land (bf16_b4096 readout 35.8 -> 32.9 us by trace);
  // the query gained nothing from it.
  constexpr int kPwADepth = NSEG == 3 ? 2 : 1;
  // weight steps in flight, up to a chunk's (a ring over two chunks' steps
  // for the readout, slots following the chunk's parity, gained nothing)
  constexpr int VPF = kPwVPF < NKL ? kPwVPF : NKL;
  constexpr int CW = 4 / KSPLIT;     // 32-column fragments per block
  static_assert(NKL % VPF == 0 && NA == 4, "ring slots fixed within a chunk");
  static_assert(NT / KQW == 32 && KQW == 16, "staging rows 32 apart");
  __shared__ f32x4 As[2 * KQW * TM];  // [stage][vector][row ^ (vector & 15)]
  const int M = A.M;
  const int m0 = blockIdx.x * TM;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int h = lane >> 5, l32 = lane & 31;
  const int wr = wave & 1, wc = (wave >> 1) % CW, kg = wave / (2 * CW);
  const int n0 = (blockIdx.y * CW + wc) * 32;  // the wave's first column
  const int nch = total_chunks(A) / 2;         // 128-k chunks
  const int last_gk = nch * NKS - 1;
  const __amdgpu_buffer_rsrc_t wres = buffer_rsrc(Wp, (int64_t)nch * KQW * Npad * 16);
  const int lo = (int)(((int64_t)h * Npad + n0 + l32) * 16);
  const int kbytes = (int)(2 * Npad * 16);  // one k step: two packed vector rows
  // k step j of this wave's share of chunk c
  auto wload = [&](f32x4& d, int c, int j) {
    const int gk = c * NKS + kg * NKL + j;
    d = buf_load(wres, lo, (gk < last_gk ? gk : last_gk) * kbytes);  // past the end: re-read the last step (unused)
  };

  // activation staging: this thread's vectors are rows tid / KQW + 32 i,
  // vector tid % KQW of each chunk
  const ASeg sg0 = seg_at(A, 0), sg1 = seg_at(A, NSEG > 1 ? 1 : 0), sg2 = seg_at(A, NSEG > 2 ? 2 : 0);
  const int c1 = sg0.nchunk / 2, c2 = c1 + (NSEG > 1 ? sg1.nchunk / 2 : 0);
  const __amdgpu_buffer_rsrc_t res0 = buffer_rsrc(sg0.p, seg_bytes(sg0, M));
  const __amdgpu_buffer_rsrc_t res1 = buffer_rsrc(sg1.p, seg_bytes(sg1, M));
  const __amdgpu_buffer_rsrc_t res2 = buffer_rsrc(sg2.p, seg_bytes(sg2, M));
  const int kin = P::KV * ((int)threadIdx.x % KQW);
  int roff0[NA], roff1[NA], roff2[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int row = m0 + ((int)threadIdx.x + i * NT) / KQW;
    roff0[i] = seg_row_off(sg0, row, M);
    roff1[i] = NSEG > 1 ? seg_row_off(sg1, row, M) : kNoLoad;
    roff2[i] = NSEG > 2 ? seg_row_off(sg2, row, M) : kNoLoad;
  }
  // rb: the second half of an fp32 source vector
  f32x4 ra[kPwADepth][NA], rb[kPwADepth][NA];
  // The bf16 segments from chunk c on, by selects (a branch between segments
  // of one type gets merged by the compiler into a dynamically indexed copy of
  // the segments in scratch memory).
  auto aload16 = [&](auto sc, int c, bool with0) {
    constexpr int S = decltype(sc)::value;
    if constexpr (NSEG == 1) {  // one segment: nothing to select
      const int kseg = c * KQW * P::KV;
#pragma unroll
      for (int i = 0; i < NA; ++i)
        load_a_raw<P, true>(res0, roff0[i], sg0.K, kseg + kin, kin, kseg * 2, ra[S][i], rb[S][i]);
      return;
    }
    const int si = (with0 && c < c1) ? 0 : (c < c2 || NSEG == 2 ? 1 : 2);
    const __amdgpu_buffer_rsrc_t res = si == 0 ? res0 : (si == 1 ? res1 : res2);
    const int kseg = (c - (si == 0 ? 0 : (si == 1 ? c1 : c2))) * KQW * P::KV;
    const int K = si == 0 ? sg0.K : (si == 1 ? sg1.K : sg2.K);
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int ro = si == 0 ? roff0[i] : (si == 1 ? roff1[i] : roff2[i]);
      load_a_raw<P, true>(res, ro, K, kseg + kin, kin, kseg * 2, ra[S][i], rb[S][i]);
    }
  };
  auto aload = [&](auto sc, int c) {  // chunk c of the whole A into register set sc
    constexpr int S = decltype(sc)::value;
    if constexpr (SRC16_0) {
      aload16(sc, c, true);
    } else if (c < c1) {  // a uniform branch to the fp32 segment's loads
      const int kseg = c * KQW * P::KV;
#pragma unroll
      for (int i = 0; i < NA; ++i)
        load_a_raw<P, false>(res0, roff0[i], sg0.K, kseg + kin, kin, kseg * 4, ra[S][i], rb[S][i]);
    } else {
      aload16(sc, c, false);
    }
  };
  const int st_base = ((int)threadIdx.x % KQW) * TM + (((int)threadIdx.x / KQW) ^ ((int)threadIdx.x % KQW));
  auto astore = [&](int stage, auto sc, int c) {  // c: the chunk the staged data belongs to
    constexpr int S = decltype(sc)::value;
    const bool s16 = SRC16_0 || c >= c1;
#pragma unroll
    for (int i = 0; i < NA; ++i)
      As[stage * KQW * TM + st_base + 32 * i] = s16 ? ra[S][i] : a_from_raw<P, false>(ra[S][i], rb[S][i]);
  };
  // fragment of k step ks (vectors 2 ks + h) for the 32 rows at r0 (a multiple of 32)
  auto afrag = [&](int stage, int ks, int r0) {
    const int v = 2 * ks + h;
    return As[stage * KQW * TM + r0 + v * TM + (l32 ^ v)];
  };
  constexpr std::integral_constant<int, 0> I0{};
  constexpr std::integral_constant<int, kPwADepth - 1> I1{};

  f32x16 acc[2] = {f32x16{}, f32x16{}};
  f32x4 ring[VPF];
#pragma unroll
  for (int p = 0; p < VPF; ++p) wload(ring[p], 0, p);
  aload(I0, 0);
  astore(0, I0, 0);
  if (nch > 1) aload(I1, 1);
  if (kPwADepth == 2 && nch > 2) aload(I0, 2);
  __syncthreads();

  const int r0 = 64 * wr, ks0 = kg * NKL;
  // the MFMAs of chunk c from LDS stage st
  auto compute = [&](int c, int st) {
    f32x4 a0 = afrag(st, ks0, r0), a1 = afrag(st, ks0, r0 + 32);
    static_for<NKL>([&](auto jc) {
      constexpr int j = decltype(jc)::value, slot = j % VPF;
      f32x4 n0 = a0, n1 = a1;
      if constexpr (j + 1 < NKL) {
        n0 = afrag(st, ks0 + j + 1, r0);
        n1 = afrag(st, ks0 + j + 1, r0 + 32);
      }
      P::mma(ring[slot], a0, acc[0]);
      P::mma(ring[slot], a1, acc[1]);
      wload(ring[slot], c + (j + VPF) / NKL, (j + VPF) % NKL);  // refill the slot, VPF steps ahead
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      a0 = n0;
      a1 = n1;
    });
  };
  if constexpr (kPwADepth == 1) {
    for (int c = 0; c < nch; ++c) {
      const int st = c & 1;
      compute(c, st);
      if (c + 1 < nch) astore(st ^ 1, I0, c + 1);
      if (c + 2 < nch) aload(I0, c + 2);
      __syncthreads();
    }
  } else {
    // two chunks per trip: set 1 holds the odd chunks, set 0 the even ones
    for (int c = 0; c < nch; c += 2) {
      compute(c, 0);
      if (c + 1 < nch) astore(1, I1, c + 1);
      if (c + 3 < nch) aload(I1, c + 3);
      __syncthreads();
      if (c + 1 >= nch) break;
      compute(c + 1, 1);
      if (c + 2 < nch) astore(0, I0, c + 2);
      if (c + 4 < nch) aload(I0, c + 4);
      __syncthreads();
    }
  }

  if constexpr (KSPLIT == 2) {  // the second group's sums to LDS, the first adds them
    float* red = (float*)As;
    if (kg == 1) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) red[(((wave - 4) * 2 + i) * 16 + r) * 64 + lane] = acc[i][r];
    }
    __syncthreads();
    if (kg == 1) return;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][r] += red[((wave * 2 + i) * 16 + r) * 64 + lane];
  }

#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int row = m0 + r0 + 32 * i + l32;
    if (row >= M) continue;
    const bool masked = ep.mask_len && (row % ep.mask_T) >= ep.mask_len[row / ep.mask_T];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j0 = n0 + 8 * q + 4 * h;
      if (j0 >= ep.N) continue;
      const f32x4 b = ep.bias ? *(const f32x4*)(ep.bias + j0) : zero4();
      f32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float v = acc[i][4 * q + e] + b[e];
        if (ep.act == 1) v = tanhf_(v);
        o[e] = masked ? 0.f : v;
      }
      if (ep.out16) {
        typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
        *(bf16x4_t*)(ep.out16 + (int64_t)row * ep.ldo + j0) = bf16x4_t{(__bf16)o[0], (__bf16)o[1], (__bf16)o[2],
                                                                         (__bf16)o[3]};
      } else {
        *(f32x4*)(ep.out + (int64_t)row * ep.ldo + j0) = o;
      }
    }
  }
}

// The weight-streaming form of a bf16 plain GEMM, if it applies (see above);
// returns false to let the caller launch the LDS-staged tile instead.
static bool try_plain_ws(const AOperand& A, const Packed& W, const PlainEpi& ep, int cus, hipStream_t st) {
  const int form = g_gemm_form.load(std::memory_order_relaxed);
  if (form == 2 || !W.bf16 || cus <= 0 || A.M <= 0 || A.nseg < 1 || A.nseg > 3 || ep.N % 4) return false;
  if (ep.defer_reduce || ep.add || ep.add2) return false;  // the caller reads the split sums; no added terms here
  for (int i = 0; i < A.nseg; ++i)
    if (A.seg[i].nchunk % 2 || (i > 0 && !A.seg[i].bf16)) return false;
  // the epilogue's vector accesses: 16-byte aligned fp32 rows and bias,
  // 8-byte aligned bf16 rows
  if (ep.ldo % 4 || (ep.bias && !aligned(ep.bias, 16)) || (ep.out16 ? !aligned(ep.out16, 8) : !aligned(ep.out, 16)))
    return false;
  // the split over K of the staged tile (small batches) stays with it
  if (form == 0 && ep.ksplit > 1) return false;
  const int nbx = ceil_div(A.M, kPwTM);
  int ksplit = (int64_t)nbx * ceil_div(ep.N, 128) < cus ? 2 : 1;
  if (form == 3 || form == 4) ksplit = form - 2;
  if (form == 0 && ksplit == 2 && (int64_t)nbx * ceil_div(ep.N, 64) < cus) return false;
  const int bn = 128 / ksplit;
  if ((int64_t)ceil_div(ep.N, bn) * bn > W.Npad) return false;  // every wave's columns inside the packed matrix
  const dim3 grid(nbx, ceil_div(ep.N, bn)), block(512);
  const bool f32_0 = !A.seg[0].bf16;
  if (A.nseg == 1 && !f32_0) {
    if (ksplit == 1)
      hipLaunchKernelGGL((k_plain_ws<1, true, 1>), grid, block, 0, st, A, W.d, W.Npad, ep);
    else
      hipLaunchKernelGGL((k_plain_ws<1, true, 2>), grid, block, 0, st, A, W.d, W.Npad, ep);
  } else if (A.nseg == 3 && f32_0) {
    if (ksplit == 1)
      hipLaunchKernelGGL((k_plain_ws<3, false, 1>), grid, block, 0, st, A, W.d, W.Npad, ep);
    else
      hipLaunchKernelGGL((k_plain_ws<3, false, 2>), grid, block, 0, st, A, W.d, W.Npad, ep);
  } else {
    return false;
  }
  g_gemm_streamed.fetch_add(1, std::memory_order_relaxed);
  return true;
}

// ------------------------------------------------ vocabulary projection

constexpr int VQMAX = 9216;             // A-tile vectors held in LDS (144 KB)

// Per precision (measured on MI355X): VTM rows per block, VNW waves, VFN
// 32-column blocks per wave step and up to VPF_MAX k groups of weight
// fragments in flight.  fp32: 64 rows, 8 waves, one block, 16 deep.  bf16
// (MFMAs 8x faster per k): 128 rows so each weight fragment feeds four
// MFMAs, and two column blocks per step so each activation fragment read
// from LDS feeds two (a 64 x 128 tile per wave, 8 MFMAs per step); 4 deep,
// as 8 deep runs out of registers.
#ifndef NMT_BF16_VTM
#define NMT_BF16_VTM 128
#endif
#ifndef NMT_BF16_VFN
#define NMT_BF16_VFN 2
#endif
#ifndef NMT_BF16_VNW
#define NMT_BF16_VNW 8
#endif
#ifndef NMT_BF16_VPF
#define NMT_BF16_VPF 4
#endif
#ifndef NMT_F32_VFN
#define NMT_F32_VFN 1
#endif
#ifndef NMT_F32_VNW
#define NMT_F32_VNW 8
#endif
#ifndef NMT_F32_VPF
#define NMT_F32_VPF 16
#endif
#ifndef NMT_VOCAB_PRIO
#define NMT_VOCAB_PRIO 1
#endif
template <class P>
struct VocabTune {
  static constexpr int VTM = P::kBF16 ? NMT_BF16_VTM : 64;
  static constexpr int VNW = P::kBF16 ? NMT_BF16_VNW : NMT_F32_VNW;
  static constexpr int VFN = P::kBF16 ? NMT_BF16_VFN : NMT_F32_VFN;
  static constexpr int VPF_MAX = P::kBF16 ? NMT_BF16_VPF : NMT_F32_VPF;
};

// Streaming vocabulary projection with an online log-sum-exp.
//
// The output bias travels inside the packed weights: rows E .. E+nb-1 of the
// packed matrix hold it (one fp32 row, or a bf16 split hi + mid + lo that
// sums to the fp32 value), and the activation rows carry 1 at those k, so
// each MFMA accumulator ends as the full logit z = t . W[:, v] + b[v].
//
// A block owns VTM rows and one slice of the vocabulary.  Its rows of the
// readout t stay in LDS for the whole kernel as 16-byte vectors
// [Kpad/KV][VTM]; the packed output weights stream straight from HBM/L2 into
// registers, VPF k groups ahead, so the main loop has no barrier.  Wave w
// takes the slice's 32-column blocks in groups of VFN (groups w, w+VNW, ...),
// each for all VTM rows.
//
// The MFMA puts the vocabulary on the output's rows and the batch rows on
// its columns, so the 16 accumulator registers of a lane are 16 logits of
// one batch row.  The fold of a group into a lane's running (max, sum) is
// then a block max (three-input maxima), one rescale of the old sum, and one
// fused multiply-add, one exp and one add per logit; a lane keeps one
// (max, sum) pair per batch row slot.  The two halves of a wave (same batch
// rows, other vocabulary rows) and the waves are merged once at the end.
// One (max, sum) pair per row and slice goes to HBM as float2 [slice][row];
// the logits never do.
//
// Slices are spread over XCDs: blocks with ids congruent mod 8 run on one
// XCD, and that XCD takes slices xcd, xcd+8, ... for every row tile, so the
// row tiles of a slice read the same weights from that XCD's L2 and the
// weights cross HBM once.
//
// Register discipline (checked in the ISA): the wave index is scalar
// (readfirstlane), loads are unconditional (clamped past the end), a ring
// slot is refilled only after its MFMAs, and A fragments ping-pong between
// two named register sets; otherwise the compiler drains every load and
// rotates registers at each loop back-edge.  No other vector-memory load is
// issued in the loop: its wait would drain the prefetch ring.
//
// PAD_LAST: the last k group of the packed matrix is all padding (no weight
// or bias row reaches it: fp32 with E + nb <= Kpad - 8), so its MFMAs, which
// would only add zeros, are skipped; its loads stay, keeping the ring's
// schedule.  With E = 500 that is 1 of 64 k groups.
template <class P, int VPF, bool PAD_LAST = false, int VTM_ = VocabTune<P>::VTM>
__global__ __launch_bounds__(VocabTune<P>::VNW * 64) void k_vocab_lse(const float* __restrict__ t, int t16, int M, int E,
                                                                      int nb, int Kpad, const f32x4* __restrict__ Wp,
                                                                      int64_t Npad, int V, int nM, int nS,
                                                                      float2* __restrict__ part,
                                                                      const int32_t* __restrict__ req1,
                                                                      const int32_t* __restrict__ req_off, int nreq,
                                                                      float* __restrict__ zreq) {
  constexpr int VTM = VTM_, VNW = VocabTune<P>::VNW, VFN = VocabTune<P>::VFN;
  constexpr int FM = VTM / 32;
  __shared__ f32x4 As[VQMAX];
  __shared__ float2 red[VNW][VTM];
  const int id = blockIdx.x, xcd = id & 7, slot = id >> 3;
  const int slice = (slot / nM) * 8 + xcd, mt = slot % nM;
  if (slice >= nS) return;
  const int m0 = mt * VTM;
  // the wave index is uniform across the wave: keep the loop control scalar
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, h = lane >> 5, l32 = lane & 31;

  const int KQ = Kpad / P::KV;

  // This slice's 32-column blocks, balanced over the slices, in groups of VFN
  // (the packed matrix has one more, all zero, past the last one with
  // columns below V).
  const int NB = (V + 31) / 32;
  const int cb_begin = (int)((int64_t)NB * slice / nS), cb_end = (int)((int64_t)NB * (slice + 1) / nS);
  const int ngrp = (cb_end - cb_begin + VFN - 1) / VFN;
  const int NKG = KQ / 2;  // k groups per column block (a multiple of VPF)

  // Running log-sum-exp of each batch row slot i (row m0 + 32 i + l32) over
  // this lane's logits: run_m the largest logit seen, run_s the sum of
  // e^(z - run_m).
  float run_m[FM], run_s[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    run_m[i] = -INFINITY;
    run_s[i] = 0.f;
  }
  // Rows that request exactly one word (req1[row], or with CSR offsets the
  // one word of a well-formed span of length 1): the lane that holds its
  // logit writes it to zreq[row] at the fold, so the combine needs no dot
  // product of its own for them.  Loaded here: no vector-memory load may be
  // issued in the loop (its wait would drain the prefetch ring).
  int rq[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int row = m0 + 32 * i + l32;
    rq[i] = -1;
    if (req1 && row < M) {
      if (!req_off) {
        rq[i] = req1[row];
      } else {
        const int j0 = req_off[row], j1 = req_off[row + 1];
        if (0 <= j0 && j1 == j0 + 1 && j1 <= nreq) rq[i] = req1[j0];
      }
    }
  }
  // The group of this slice whose MFMAs produce each slot's requested logit
  // in this lane (column 32 cb + acc_row(r, h) sits in lane half h when bit 2
  // of the column is h), or -1: the loop then tests one integer per slot.
  int rq_g[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int cb = rq[i] >> 5;
    rq_g[i] = (rq[i] >= 0 && cb >= cb_begin && cb < cb_end && ((rq[i] >> 2) & 1) == h) ? (cb - cb_begin) / VFN : -1;
  }

  // Weight fragments are read through a buffer resource over the packed
  // matrix: a lane's offset (its column and k half) is fixed, and one scalar
  // offset per step selects the group's k group, so a step costs one scalar
  // add and no address arithmetic.  Ring slot p always holds step q with
  // q % VPF == p; the last VPF steps of a group refill the ring with the
  // first VPF steps of the wave's next group.  A wave past its last group,
  // or a group's missing last block, reads other columns of the matrix
  // (masked at the fold); offsets past the end of the matrix read zeros.
  const __amdgpu_buffer_rsrc_t wres =
      __builtin_amdgcn_make_buffer_rsrc((void*)Wp, (short)0, (int)(KQ * Npad * 16), 0x00020000);
  const int kbytes = (int)(32 * Npad);             // one k group: two rows of vectors
  int lane_off[VFN];
#pragma unroll
  for (int f = 0; f < VFN; ++f) lane_off[f] = (int)((h * Npad + l32 + 32 * f) * 16);
  auto gbase = [&](int g) { return g < ngrp ? (cb_begin + g * VFN) * 512 : 0; };  // bytes of the group's block 0
  auto load = [&](f32x4 (&dst)[VFN], int soff) {
#pragma unroll
    for (int f = 0; f < VFN; ++f)
      dst[f] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(wres, lane_off[f], soff, 0));
  };
  int sbase = gbase(wave);  // the group whose steps are being loaded
  f32x4 ring[VPF][VFN];
#pragma unroll
  for (int p = 0; p < VPF; ++p) load(ring[p], sbase + p * kbytes);

  // Stationary activation tile: As[kq][m] = vector kq of row m0 + m, with
  // the bias slots set to 1.  Staged after the first weight loads went out,
  // so their latency and the tile's overlap.
  for (int idx = threadIdx.x; idx < KQ * VTM; idx += VNW * 64) {
    const int m = idx % VTM, kq = idx / VTM, row = m0 + m;
    As[kq * VTM + m] = with_bias_ones<P>(
        load_a_vec<P>(row >= M ? nullptr
                      : t16    ? (const char*)((const __bf16*)t + (int64_t)row * bf16_row(E))
                               : (const char*)(t + (int64_t)row * E),
                      t16, E, kq * P::KV),
        kq, E, nb);
  }
  __syncthreads();
  const f32x4* arow = As + h * VTM + l32;  // + 2*kg*VTM per k group
  f32x4 ae[FM], ao[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) ae[i] = arow[32 * i];
  static_assert(VPF % 2 == 0, "even/odd fragment sets");

  // groups wave, wave + VNW, ... of the slice
  for (int gcur = wave; gcur < ngrp; gcur += VNW) {
    f32x16 acc[FM][VFN];
    const int nbase = gbase(gcur + VNW);
    // One k-group step; `zc` (compile time) starts the accumulators from an
    // inline zero instead of clearing them with register moves; `soff` is
    // the scalar offset of the step that refills this slot; `ablk` is the
    // LDS address of k group kg0 + 1 for the block starting at kg0, so the
    // next step's fragments sit at compile-time offsets from it (the last
    // step of a group wraps to k group 0 of the next one).
    auto kstep = [&](const f32x4* ablk, auto pc, auto zc, auto last_blk, int soff) {
      constexpr int p = decltype(pc)::value;
      const f32x4* an = (decltype(last_blk)::value && p == VPF - 1) ? arow : ablk + p * 2 * VTM;
      f32x4 a[FM];
      if constexpr (p % 2 == 0) {
#pragma unroll
        for (int i = 0; i < FM; ++i) {
          ao[i] = an[32 * i];
          a[i] = ae[i];
        }
      } else {
#pragma unroll
        for (int i = 0; i < FM; ++i) {
          ae[i] = an[32 * i];
          a[i] = ao[i];
        }
      }
      // weights as the MFMA's row operand, activations as its column operand
      constexpr bool pad_step = PAD_LAST && decltype(last_blk)::value && p == VPF - 1;
      if constexpr (!pad_step) {
#pragma unroll
        for (int f = 0; f < VFN; ++f)
#pragma unroll
          for (int i = 0; i < FM; ++i) {
            if constexpr (decltype(zc)::value)
              acc[i][f] = P::mma0(ring[p][f], a[i]);
            else
              P::mma(ring[p][f], a[i], acc[i][f]);
          }
      }
      load(ring[p], soff);  // refill the slot just consumed, VPF steps ahead
      // Instruction order within the step: one MFMA, the next step's A
      // fragment reads (so they have the remaining MFMAs to land), the rest
      // of the MFMAs, then the refill.
      if constexpr (!pad_step) {
        constexpr int kMfmaPerStep = FM * VFN * (P::kBF16 ? 1 : 4);  // fp32: four MFMAs per fragment pair
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, FM, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, kMfmaPerStep - 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, VFN, 0);
      }
    };
    // Blocks of VPF steps (a group has at least two): the first starts from
    // zero, the last refills the ring from the next group.  MFMA steps run at raised priority and the
    // fold at normal priority, so the other wave on the SIMD keeps issuing
    // MFMAs while this one folds.
    __builtin_amdgcn_s_setprio(NMT_VOCAB_PRIO);
    static_for<VPF>([&](auto pc) {
      constexpr int p = decltype(pc)::value;
      kstep(arow + 2 * VTM, pc, std::bool_constant<p == 0>{}, std::false_type{}, sbase + (VPF + p) * kbytes);
    });
    for (int kg0 = VPF; kg0 < NKG - VPF; kg0 += VPF) {
      const int s0 = sbase + (kg0 + VPF) * kbytes;
      const f32x4* ablk = arow + (kg0 + 1) * 2 * VTM;
      static_for<VPF>([&](auto pc) {
        constexpr int p = decltype(pc)::value;
        kstep(ablk, pc, std::false_type{}, std::false_type{}, s0 + p * kbytes);
      });
    }
    {
      const f32x4* ablk = arow + (NKG - VPF + 1) * 2 * VTM;
      static_for<VPF>([&](auto pc) {
        constexpr int p = decltype(pc)::value;
        kstep(ablk, pc, std::false_type{}, std::true_type{}, nbase + p * kbytes);
      });
    }
    __builtin_amdgcn_s_setprio(0);
    sbase = nbase;

    // Register r of a lane holds vocabulary row 32 cb + acc_row(r, h).  A
    // group with columns past V or missing blocks (only at the end of a
    // slice) masks them out; the test is uniform over the wave.
    const int cb0 = cb_begin + gcur * VFN;
    if ((cb0 + VFN) * 32 > V || cb0 + VFN > cb_end) {
#pragma unroll
      for (int f = 0; f < VFN; ++f)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const bool ok = cb0 + f < cb_end && (cb0 + f) * 32 + acc_row(r, h) < V;
#pragma unroll
          for (int i = 0; i < FM; ++i) acc[i][f][r] = ok ? acc[i][f][r] : -INFINITY;
        }
    }
    // A requested column in this group: column 32 (cb0 + f) + acc_row(r, h)
    // sits in register r of block f of lane half h.  Only the group's blocks
    // below cb_end are this slice's (the rest belong to the next slice and
    // were masked above), so every column has exactly one writer; columns
    // past V are never requested by a valid id.  A wave-uniform branch, taken
    // only when some lane of the wave holds a requested logit here (the
    // per-lane test alone was if-converted into some 400 mask and select
    // instructions per group, with SGPR spills into vector lanes).
    bool hit = false;
#pragma unroll
    for (int i = 0; i < FM; ++i) hit |= rq_g[i] == gcur;
    if (__builtin_amdgcn_ballot_w64(hit)) {
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        if (rq_g[i] == gcur) {
          const int d = rq[i] - 32 * cb0;
          const int idx = (d >> 5) * 16 + ((d & 31) >> 3) * 4 + (d & 3);  // 16 f + r
          float z = 0.f;
#pragma unroll
          for (int f = 0; f < VFN; ++f)
#pragma unroll
            for (int r = 0; r < 16; ++r) z = idx == 16 * f + r ? acc[i][f][r] : z;
          zreq[m0 + 32 * i + l32] = z;
        }
      }
    }
    // fold the group into each row slot's running log-sum-exp
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      float bm = acc[i][0][0];
#pragma unroll
      for (int f = 0; f < VFN; ++f)
#pragma unroll
        for (int r = 0; r < 16; ++r) bm = fmaxf(bm, acc[i][f][r]);
      const float mn = fmaxf(run_m[i], bm);
      const bool none = mn == -INFINITY;  // nothing but masked logits so far
      const float sc = none ? 1.f : __builtin_amdgcn_exp2f((run_m[i] - mn) * kLog2e);
      const float nm = none ? 0.f : -mn * kLog2e;
      float s0 = 0.f, s1 = 0.f;
#pragma unroll
      for (int f = 0; f < VFN; ++f)
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          s0 += __builtin_amdgcn_exp2f(fmaf(acc[i][f][r], kLog2e, nm));
          s1 += __builtin_amdgcn_exp2f(fmaf(acc[i][f][r + 1], kLog2e, nm));
        }
      run_s[i] = fmaf(run_s[i], sc, s0 + s1);
      run_m[i] = mn;
    }
  }

  // merge the two halves of the wave (lanes l32 and l32 + 32 hold the same rows)
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const float om = __shfl_xor(run_m[i], 32, 64), os = __shfl_xor(run_s[i], 32, 64);
    const float mx = fmaxf(run_m[i], om);
    float s = 0.f;
    if (mx != -INFINITY)
      s = run_s[i] * __builtin_amdgcn_exp2f((run_m[i] - mx) * kLog2e) +
          os * __builtin_amdgcn_exp2f((om - mx) * kLog2e);
    if (h == 0) red[wave][32 * i + l32] = float2{mx, s};
  }
  __syncthreads();
  // merge the waves and write this slice's partial for each row
  for (int rl = threadIdx.x; rl < VTM; rl += VNW * 64) {
    const int row = m0 + rl;
    float mx = -INFINITY;
#pragma unroll
    for (int w = 0; w < VNW; ++w) mx = fmaxf(mx, red[w][rl].x);
    float s = 0.f;
    if (mx != -INFINITY) {
#pragma unroll
      for (int w = 0; w < VNW; ++w) {
        const float mw = red[w][rl].x;
        if (mw != -INFINITY) s += red[w][rl].y * __builtin_amdgcn_exp2f((mw - mx) * kLog2e);
      }
    }
    // (max logit, sum of e^(z - max)) in natural-log units
    if (row < M) part[(int64_t)slice * M + row] = float2{mx, s};
  }
}

// Slices per row tile: the multiple of 8 (one per XCD) whose launch finishes
// first.  A block holds one CU, so a launch of nM x nS blocks runs in
// ceil(nM nS / CUs) rounds, each as long as one block: NB / nS column blocks
// plus a fixed cost (staging the activation tile, the final merge) of about
// kVocabBlockFixed column blocks.  Batches whose row tiles divide the CUs
// evenly get one round (2000 rows: 8 slices); the others, more rounds of
// shorter blocks (1445 rows: 32 slices in three rounds instead of 16 in
// two, 25 % less time).
constexpr int kVocabBlockFixed = 4;
// nmt_score_workspace_bytes takes its maximum over multiples of 32 rows.
static_assert(VocabTune<PrecF32>::VTM % 32 == 0 && VocabTune<PrecBF16>::VTM % 32 == 0 && kPlainSmallTM % 32 == 0,
              "row tiles in whole multiples of 32");
constexpr int kVocabMaxSlices = 256;
// Small fp32 batches (the levels of a forest, the shrinking phrase loop) may
// take row tiles of 32: the launch's blocks then split the rows finer, so the
// SIMDs of a block end closer together (a SIMD's share of a block is whole
// 32 x 32 groups instead of 64 x 32 ones) and less row padding is computed;
// each weight fragment feeds half the MFMAs, so 32 k groups stay in flight.
// That form exists for the deepest prefetch with a skipped padding k group
// (the paper's E = 500), its one instantiation.
constexpr int kVocabSmallM = 768, kVocabSmallTM = 32, kVocabSmallVPF = 32;

// Launch time of nM row tiles in nS slices, in the time of one column block
// of the tile: rounds of one block per CU, each as long as one block.  With
// by_simd a block lasts as long as its busiest SIMD's whole groups (four
// SIMDs share a block's groups); otherwise its share of the columns, the
// model the 64-row tiles' slice counts were chosen and measured by.
static double vocab_cost(int nM, int nS, int NB, int cus, double fixed, bool by_simd) {
  const double rounds = (double)ceil_div((int64_t)nM * nS, cus);
  const double block = by_simd ? 4.0 * ceil_div(ceil_div(NB, nS), 4) : (double)NB / nS;
  return rounds * (block + fixed);
}

int vocab_slices(int M, int V, bool bf16, int cus, int tm) {
  const int nM = ceil_div(M, tm);
  const int NB = (V + 31) / 32;
  // a block's fixed costs, in the time of one of its column blocks
  const double fixed = tm < 64 ? 2.0 * kVocabBlockFixed : kVocabBlockFixed;
  int best = 8;
  double best_cost = 0;
  for (int nS = 8; nS <= kVocabMaxSlices && (nS == 8 || nS <= NB); nS += 8) {
    const double cost = vocab_cost(nM, nS, NB, cus, fixed, tm < 64);
    if (nS == 8 || cost < best_cost) {
      best_cost = cost;
      best = nS;
    }
  }
  return best;
}

// The row tile of a launch: 32 where that form exists and the launch's
// time by whole groups per SIMD beats the 64-row tile's (in equal units;
// measured on the phrase loop's levels: 500, 232 and 125 rows 2-8 % faster,
// 364 rows slower, as this predicts).
int vocab_tm(int M, int V, bool bf16, int64_t Kpad, int E, int nb, int cus) {
  if (bf16) return VocabTune<PrecBF16>::VTM;
  constexpr int TM = VocabTune<PrecF32>::VTM;
  const int64_t nkg = Kpad / (2 * PrecF32::KV);
  const bool fits = nkg % kVocabSmallVPF == 0 && nkg >= 2 * kVocabSmallVPF && E + nb <= Kpad - 2 * PrecF32::KV;
  if (M > kVocabSmallM || !fits) return TM;
  const int NB = (V + 31) / 32;
  const double small = vocab_cost(ceil_div(M, kVocabSmallTM), vocab_slices(M, V, false, cus, kVocabSmallTM), NB,
                                  cus, 2.0 * kVocabBlockFixed, true);
  const double large = (double)TM / kVocabSmallTM *
                       vocab_cost(ceil_div(M, TM), vocab_slices(M, V, false, cus, TM), NB, cus, kVocabBlockFixed, true);
  return small < large ? kVocabSmallTM : TM;
}

// The vocabulary kernel addresses the packed weights with 32-bit byte offsets.
bool vocab_offsets_fit(int64_t Kpad, int64_t Npad, bool bf16) {
  return Kpad / (bf16 ? PrecBF16::KV : PrecF32::KV) * Npad * 16 < ((int64_t)1 << 31);
}

int vocab_max_kpad(bool bf16) {
  return bf16 ? VQMAX / VocabTune<PrecBF16>::VTM * PrecBF16::KV : VQMAX / VocabTune<PrecF32>::VTM * PrecF32::KV;
}

template <class P>
hipError_t vocab_lse(const float* t, int t16, int M, int E, const Packed& W, int V, float2* part, int nS, int tm,
                     const int32_t* req1, const int32_t* req_off, int nreq, float* zreq, hipStream_t st) {
  const int nkg = (int)(W.Kpad / (2 * P::KV));
  const f32x4* Wp = (const f32x4*)W.d;
  if constexpr (!P::kBF16) {
    if (tm == kVocabSmallTM) {
      const int nM = ceil_div(M, kVocabSmallTM);
      hipLaunchKernelGGL((k_vocab_lse<P, kVocabSmallVPF, true, kVocabSmallTM>), dim3((unsigned)(nS / 8 * 8 * nM)),
                         dim3(VocabTune<P>::VNW * 64), 0, st, t, t16, M, E, W.nbias, (int)W.Kpad, Wp, W.Npad, V, nM,
                         nS, part, req1, req_off, nreq, zreq);
      return hipGetLastError();
    }
  }
  const int nM = ceil_div(M, VocabTune<P>::VTM);
  dim3 grid((unsigned)(nS / 8 * 8 * nM)), block(VocabTune<P>::VNW * 64);
  constexpr int PF = VocabTune<P>::VPF_MAX;
  // the deepest prefetch that divides the k groups into at least two blocks
  auto fits = [&](int vpf) { return PF >= vpf && nkg % vpf == 0 && nkg >= 2 * vpf; };
  // the last k group only padding (see PAD_LAST; taken with the deepest prefetch)
  const bool pad_last = !P::kBF16 && E + W.nbias <= W.Kpad - 2 * P::KV;
  if (fits(16) && pad_last)
    hipLaunchKernelGGL((k_vocab_lse<P, (PF >= 16 ? 16 : 2), !P::kBF16>), grid, block, 0, st, t, t16, M, E, W.nbias,
                       (int)W.Kpad, Wp, W.Npad, V, nM, nS, part, req1, req_off, nreq, zreq);
  else if (fits(16))
    hipLaunchKernelGGL((k_vocab_lse<P, (PF >= 16 ? 16 : 2)>), grid, block, 0, st, t, t16, M, E, W.nbias, (int)W.Kpad, Wp,
                       W.Npad, V, nM, nS, part, req1, req_off, nreq, zreq);
  else if (fits(8))
    hipLaunchKernelGGL((k_vocab_lse<P, (PF >= 8 ? 8 : 2)>), grid, block, 0, st, t, t16, M, E, W.nbias, (int)W.Kpad, Wp,
                       W.Npad, V, nM, nS, part, req1, req_off, nreq, zreq);
  else if (fits(4))
    hipLaunchKernelGGL((k_vocab_lse<P, 4>), grid, block, 0, st, t, t16, M, E, W.nbias, (int)W.Kpad, Wp, W.Npad, V, nM, nS,
                       part, req1, req_off, nreq, zreq);
  else if (fits(2))
    hipLaunchKernelGGL((k_vocab_lse<P, 2>), grid, block, 0, st, t, t16, M, E, W.nbias, (int)W.Kpad, Wp, W.Npad, V, nM, nS,
                       part, req1, req_off, nreq, zreq);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_vocab_lse(const float* t, int t16, int M, int E, const Packed& W, int V, float2* part, int nS,
                            int tm, const int32_t* req1, const int32_t* req_off, int nreq, float* zreq,
                            hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (t16 && !W.bf16) return hipErrorInvalidValue;
  // the small tile only where its form exists (see vocab_tm)
  const int64_t nkg = W.Kpad / (2 * (W.bf16 ? PrecBF16::KV : PrecF32::KV));
  if (tm == kVocabSmallTM && (W.bf16 || nkg % kVocabSmallVPF || nkg < 2 * kVocabSmallVPF ||
                              E + W.nbias > W.Kpad - 2 * PrecF32::KV))
    return hipErrorInvalidValue;
  if (W.Kpad > vocab_max_kpad(W.bf16) || W.Krows != E || W.nbias < 1 || W.Npad < ((int64_t)V + 31) / 32 * 32 + 32)
    return hipErrorInvalidValue;
  if (!vocab_offsets_fit(W.Kpad, W.Npad, W.bf16)) return hipErrorInvalidValue;
  if (req1 && !zreq) return hipErrorInvalidValue;
  return W.bf16 ? vocab_lse<PrecBF16>(t, t16, M, E, W, V, part, nS, tm, req1, req_off, nreq, zreq, st)
                : vocab_lse<PrecF32>(t, 0, M, E, W, V, part, nS, tm, req1, req_off, nreq, zreq, st);
}

// ---------------------------------------------------- partials combine

// Dot product of two 16-byte vectors in precision P (fp32 accumulation).
template <class P>
__device__ __forceinline__ float dot_vec(const f32x4& a, const f32x4& b) {
  if constexpr (P::kBF16) {
    const bf16x8 x = __builtin_bit_cast(bf16x8, a), y = __builtin_bit_cast(bf16x8, b);
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) s += (float)x[e] * (float)y[e];
    return s;
  } else {
    return a[0] * b[0] + a[1] * b[1] + a[2] * b[2] + a[3] * b[3];
  }
}

// One wave per row: merges the per-slice (max, sum) pairs into logZ, scores
// each requested word with its own dot product over the packed column of w,
// bias rows included (t rounded, and 1 at the bias slots, as the vocabulary
// kernel's MFMA inputs are), and checks the row's ids.  A row with any id out of range, or with malformed request
// offsets, gets NaN outputs and sets the flag.
template <class P>
__global__ __launch_bounds__(256) void k_lse_combine(int B, const float2* __restrict__ part, int nS,
                                                     const float* __restrict__ t, int t16, int E, int nb, int Kpad,
                                                     const f32x4* __restrict__ Wp, int64_t Npad, int V,
                                                     Requests rq,
                                                     const int32_t* __restrict__ y_prev,
                                                     const int32_t* __restrict__ sent_id, int S, float* logp,
                                                     float* logZ, int* err, const float* __restrict__ zreq) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= B) return;
  // Every load that depends on no other is issued before any is used, so the
  // kernel waits for one round trip to memory instead of a chain of them: the
  // row's ids, its first 64 partials, its requested logit, and (one request
  // per row, no offsets) its requested word.
  const int y = y_prev[row], s = sent_id[row];
  const int sr = rq.state_row ? rq.state_row[row] : 0;
  const float2 p0 = lane < nS ? part[(int64_t)lane * B + row] : make_float2(-INFINITY, 0.f);
  const float zr = zreq ? zreq[row] : 0.f;
  const int w_row = rq.req_off ? 0 : rq.req[row];
  const int j0 = rq.req_off ? rq.req_off[row] : row, j1 = rq.req_off ? rq.req_off[row + 1] : row + 1;
  const bool span_ok = 0 <= j0 && j0 <= j1 && j1 <= rq.nreq;
  bool ok = span_ok && y >= -1 && y < V && s >= 0 && s < S;
  if (rq.state_row) ok = ok && sr >= 0 && sr < rq.pool_rows;
  if (!rq.req_off)
    ok = ok && w_row >= 0 && w_row < V;
  else if (span_ok)
    for (int j = j0; j < j1; ++j) ok = ok && rq.req[j] >= 0 && rq.req[j] < V;
  if (!ok) {
    if (lane == 0) {
      if (span_ok)
        for (int j = j0; j < j1; ++j) logp[j] = __builtin_nanf("");
      if (logZ) logZ[row] = __builtin_nanf("");
      atomicOr(err, 1);
    }
    return;
  }
  // the same arithmetic, in the same order, as a lane-strided pass over the slices
  float mx = fmaxf(-INFINITY, p0.x);
  for (int i = lane + 64; i < nS; i += 64) mx = fmaxf(mx, part[(int64_t)i * B + row].x);
  mx = wave_max(mx);
  float sum = 0.f;
  if (p0.x != -INFINITY) sum += p0.y * expf(p0.x - mx);
  for (int i = lane + 64; i < nS; i += 64) {
    const float2 p = part[(int64_t)i * B + row];
    if (p.x != -INFINITY) sum += p.y * expf(p.x - mx);
  }
  sum = wave_sum(sum);
  const float lz = mx + logf(sum);
  if (lane == 0 && logZ) logZ[row] = lz;
  if (zreq && j1 == j0 + 1) {  // one request: its logit taken by the vocabulary kernel
    if (lane == 0) logp[j0] = zr - lz;
    return;
  }
  const char* tr = t16 ? (const char*)((const __bf16*)t + (int64_t)row * bf16_row(E))
                       : (const char*)(t + (int64_t)row * E);
  for (int j = j0; j < j1; ++j) {
    const int w = rq.req[j];
    float dot = 0.f;
    for (int kq = lane; kq < Kpad / P::KV; kq += 64)
      dot += dot_vec<P>(with_bias_ones<P>(load_a_vec<P>(tr, t16, E, kq * P::KV), kq, E, nb),
                        Wp[(int64_t)kq * Npad + w]);
    dot = wave_sum(dot);
    if (lane == 0) logp[j] = dot - lz;
  }
}

hipError_t launch_lse_combine(int B, const float2* part, int nS, const float* t, int t16, int E, const Packed& W, int V,
                              const Requests& rq, const int32_t* y_prev,
                              const int32_t* sent_id, int S, float* logp, float* logZ, int* err, const float* zreq, hipStream_t st) {
  if (B <= 0) return hipSuccess;
  if (W.Krows != E || W.nbias < 1 || (t16 && !W.bf16)) return hipErrorInvalidValue;
  if (W.bf16)
    hipLaunchKernelGGL(k_lse_combine<PrecBF16>, dim3(ceil_div(B, 4)), dim3(256), 0, st, B, part, nS, t, t16, E,
                       W.nbias, (int)W.Kpad, (const f32x4*)W.d, W.Npad, V, rq, y_prev, sent_id, S, logp, logZ, err, zreq);
  else
    hipLaunchKernelGGL(k_lse_combine<PrecF32>, dim3(ceil_div(B, 4)), dim3(256), 0, st, B, part, nS, t, 0, E,
                       W.nbias, (int)W.Kpad, (const f32x4*)W.d, W.Npad, V, rq, y_prev, sent_id, S, logp, logZ, err, zreq);
  return hipGetLastError();
}

// ------------------------------------------------------------ attention

// Attention scores.  With tanh x = 1 - 2 / (e^{2x} + 1) and
// e^{2(k+q)} = 2^{ck} 2^{cq} (c = 2 log2 e),
//   e_i = v . tanh(k_i + q) = sum(v) + sum_a (-2 v_a) / (2^{c k_ia} 2^{c q_a} + 1),
// and the softmax over i ignores the constant sum(v).  The keys' factors
// K = 2^{c k} are formed once per source position when the source is
// encoded, the query's Q = 2^{c q} once per row, so the kernels score
//   e'_i = sum_a w_a / (K_ia Q_a + 1)   with w = -2 v:
// one fma, the hardware reciprocal and one fma per term (one
// transcendental instead of an exp and a reciprocal).
//
// A factor is a finite fp32 number only while |c x| < 128, so the factor
// exponents are clamped to [-126, 126].  The product K Q is then the exact
// 2^{c(k+q)} (up to rounding; it over- or underflows only where tanh has
// saturated) as long as neither exponent was clamped.  It stays exact to
// within 2^-26 of a term when one exponent is clamped and the other is at
// most kFactorSafe in magnitude: then |c(k+q)| > 26 in both the true and
// the clamped product, where the term is 0 or w to that precision.  Only
// when a clamped exponent meets an opposite one above kFactorSafe can the
// clamp change a term (k = 50, q = -49.5 would score tanh 0 instead of
// tanh 0.5).  So each source sentence carries a flag, set when the
// magnitude of any of its key exponents exceeds kFactorSafe, and each
// attention tile tests its queries the same way; a tile with both scores
// every term as w / (2^{c(k+q)} + 1) from the keys themselves (an exp2 and
// a reciprocal per term), which is exact for any k and q.
constexpr float kTanhScale = 2.f * kLog2e;
constexpr float kFactorSafe = 100.f;
__device__ __forceinline__ float tanh_factor(float x) {
  return __builtin_amdgcn_exp2f(fminf(fmaxf(x * kTanhScale, -126.f), 126.f));
}
__device__ __forceinline__ f32x4 tanh_factor(f32x4 x) {
  return f32x4{tanh_factor(x[0]), tanh_factor(x[1]), tanh_factor(x[2]), tanh_factor(x[3])};
}
// True when some factor exponent of x is beyond kFactorSafe.
__device__ __forceinline__ bool factor_big(f32x4 x) {
  const float m = fmaxf(fmaxf(fabsf(x[0]), fabsf(x[1])), fmaxf(fabsf(x[2]), fabsf(x[3])));
  return m * kTanhScale > kFactorSafe;
}
__device__ __forceinline__ float score_term(float kf, float qf, float w, float acc) {
  return fmaf(w, __builtin_amdgcn_rcpf(fmaf(kf, qf, 1.f)), acc);
}
// The same term from the key k and the query q themselves: exact for any
// magnitudes (2^{c(k+q)} is inf or 0 exactly where tanh has saturated).
__device__ __forceinline__ float score_term_exact(float k, float q, float w, float acc) {
  return fmaf(w, __builtin_amdgcn_rcpf(__builtin_amdgcn_exp2f((k + q) * kTanhScale) + 1.f), acc);
}
template <bool EXACT>
__device__ __forceinline__ float score_term_t(float k, float q, float w, float acc) {
  return EXACT ? score_term_exact(k, q, w, acc) : score_term(k, q, w, acc);
}

// Four context values at element index i of c: fp32, or (c_bf16) bf16
// rounded to nearest even, the rounding the bf16 GEMMs apply when they
// stage an fp32 operand.
__device__ __forceinline__ void store_c4(float* c, int64_t i, const f32x4& v, int c_bf16) {
  if (c_bf16) {
    typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
    *(bf16x4_t*)((__bf16*)c + i) = bf16x4_t{(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
  } else {
    *(f32x4*)(c + i) = v;
  }
}

// The keys' factors of one sentence per block, and the sentence's flag: 1
// when some key exponent exceeds kFactorSafe in magnitude (the positions
// past the length hold zero keys).
__global__ __launch_bounds__(1024) void k_key_factors(int64_t per_sentence4, const f32x4* __restrict__ x,
                                                      f32x4* __restrict__ out, int32_t* __restrict__ big) {
  const int64_t base = (int64_t)blockIdx.x * per_sentence4;
  bool b = false;
  for (int64_t i = threadIdx.x; i < per_sentence4; i += 1024) {
    const f32x4 v = x[base + i];
    b |= factor_big(v);
    out[base + i] = tanh_factor(v);
  }
  b = __syncthreads_or(b);
  if (threadIdx.x == 0) big[blockIdx.x] = b ? 1 : 0;
}

hipError_t launch_key_factors(int S, int Tpad, int A, const float* pctx, float* kfac, int32_t* big, hipStream_t st) {
  if (S <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_key_factors, dim3(S), dim3(1024), 0, st, (int64_t)Tpad * A / 4, (const f32x4*)pctx,
                     (f32x4*)kfac, big);
  return hipGetLastError();
}

// Fallback for more sentences than the grouping kernel counts: one block
// (4 waves) per row.  Wave w scores source positions w, w+4, ... (each lane
// covers float4 pieces of the attention width), the block normalises the
// scores over the row's sentence length, then every thread accumulates
// float4 pieces of the context over the unmasked positions.
template <int NQ>
__global__ __launch_bounds__(256) void k_attention(int B, int A, int C, int Tpad, QuerySrc q,
                                                   const float* __restrict__ kfac, const float* __restrict__ pctx,
                                                   const int32_t* __restrict__ kbig, const float* __restrict__ ctx,
                                                   const int32_t* __restrict__ len,
                                                   const int32_t* __restrict__ sent_id, int S,
                                                   const float* __restrict__ v, float* __restrict__ c,
                                                   float* __restrict__ alpha, int c_bf16) {
  __shared__ float e[kMaxTpad];
  __shared__ float red[8];
  const int row = blockIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int s = sent_id[row];
  if (s < 0 || s >= S) {  // flagged and NaN-ed by the combine kernel; keep the rest finite
    for (int k4 = threadIdx.x; k4 < C / 4; k4 += 256) store_c4(c, (int64_t)row * C + 4 * k4, zero4(), c_bf16);
    if (alpha)
      for (int i = threadIdx.x; i < Tpad; i += 256) alpha[(int64_t)row * Tpad + i] = 0.f;
    return;
  }
  const int L = len[s];
  const int A4 = A / 4;
  f32x4 qv[NQ], vv[NQ];  // the query and weights -2 v (see score_term)
  bool big = false;
#pragma unroll
  for (int k = 0; k < NQ; ++k) {
    const int a4 = lane + 64 * k;
    qv[k] = a4 < A4 ? load_q(q, row, A, a4) : zero4();
    vv[k] = a4 < A4 ? *(const f32x4*)(v + 4 * a4) * -2.f : zero4();
    big |= factor_big(qv[k]);
  }
  // Every wave holds the row's whole query, so the test is uniform over the block.
  const bool exact = __any(big) && kbig[s];
  auto score = [&](auto exact_tag, const float* P) {
    constexpr bool EX = decltype(exact_tag)::value;
    for (int i = wave; i < L; i += 4) {
      float acc = 0.f;
#pragma unroll
      for (int k = 0; k < NQ; ++k) {
        const int a4 = lane + 64 * k;
        if (a4 < A4) {
          const f32x4 p = *(const f32x4*)(P + (int64_t)i * A + 4 * a4);
#pragma unroll
          for (int x = 0; x < 4; ++x) acc = score_term_t<EX>(p[x], qv[k][x], vv[k][x], acc);
        }
      }
      acc = wave_sum(acc);
      if (lane == 0) e[i] = acc;
    }
  };
  if (exact) {
    score(std::true_type{}, pctx + (int64_t)s * Tpad * A);
  } else {
#pragma unroll
    for (int k = 0; k < NQ; ++k) qv[k] = tanh_factor(qv[k]);  // padding lanes: factor 1, weight 0
    score(std::false_type{}, kfac + (int64_t)s * Tpad * A);
  }
  __syncthreads();
  float mx = -INFINITY;
  for (int i = threadIdx.x; i < L; i += 256) mx = fmaxf(mx, e[i]);
  mx = wave_max(mx);
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  float sum = 0.f;
  for (int i = threadIdx.x; i < L; i += 256) sum += expf(e[i] - mx);
  sum = wave_sum(sum);
  if (lane == 0) red[4 + wave] = sum;
  __syncthreads();
  const float inv = 1.f / ((red[4] + red[5]) + (red[6] + red[7]));
  for (int i = threadIdx.x; i < L; i += 256) e[i] = expf(e[i] - mx) * inv;
  if (alpha)
    for (int i = threadIdx.x; i < Tpad; i += 256) alpha[(int64_t)row * Tpad + i] = 0.f;
  __syncthreads();
  if (alpha)
    for (int i = threadIdx.x; i < L; i += 256) alpha[(int64_t)row * Tpad + i] = e[i];
  const float* X = ctx + (int64_t)s * Tpad * C;
  for (int k4 = threadIdx.x; k4 < C / 4; k4 += 256) {
    f32x4 acc = zero4();
    for (int i = 0; i < L; ++i) {
      const f32x4 x = *(const f32x4*)(X + (int64_t)i * C + 4 * k4);
      const float a = e[i];
      acc[0] += a * x[0];
      acc[1] += a * x[1];
      acc[2] += a * x[2];
      acc[3] += a * x[3];
    }
    store_c4(c, (int64_t)row * C + 4 * k4, acc, c_bf16);
  }
}

// Rows grouped by sentence, so that a block scores up to G rows of one
// sentence and reads that sentence's keys and annotations once for all of
// them.  k_group_rows (one block) counts the rows of each sentence in LDS
// (rows with an invalid sentence id go to an extra bucket, scored as zeros),
// orders the sentences longest first, lists the rows sentence by sentence
// in that order in perm, and cuts each sentence's rows into tiles (sentence
// or -1, first index into perm, row count).  A tile's work grows with its
// sentence's length, and the blocks are dispatched in tile order, so the
// longest tiles start first and the short ones fill the slots that free up
// (a sentence-order list left a second round of a few long tiles).  The
// order of rows inside a sentence does not matter: each row's arithmetic is
// the same in any tile.
// Exclusive prefix sums over the 1024 threads of a block of two values per
// thread (wave scans with shuffles, then one scan of the 16 wave totals);
// returns the block totals.  wsum: 2 x 16 ints of LDS, free on entry and
// on return.
__device__ __forceinline__ int2 block_scan2(int& a, int& b, int (*wsum)[16]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = a, y = b;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int px = __shfl_up(x, o, 64), py = __shfl_up(y, o, 64);
    if (lane >= o) {
      x += px;
      y += py;
    }
  }
  if (lane == 63) {
    wsum[0][wave] = x;
    wsum[1][wave] = y;
  }
  __syncthreads();
  if (wave == 0) {
    int u = lane < 16 ? wsum[0][lane] : 0, w = lane < 16 ? wsum[1][lane] : 0;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      const int pu = __shfl_up(u, o, 64), pw = __shfl_up(w, o, 64);
      if (lane >= o) {
        u += pu;
        w += pw;
      }
    }
    if (lane < 16) {
      wsum[0][lane] = u;
      wsum[1][lane] = w;
    }
  }
  __syncthreads();
  const int2 tot = make_int2(wsum[0][15], wsum[1][15]);
  a = (wave ? wsum[0][wave - 1] : 0) + x - a;
  b = (wave ? wsum[1][wave - 1] : 0) + y - b;
  __syncthreads();
  return tot;
}

constexpr int kGroupRowsHeld = 8;  // rows per thread whose bucket stays in registers

struct GroupScratch {
  int cnt[kGroupMaxS + 1];    // rows per bucket, then the bucket's write cursor
  int order[kGroupMaxS + 1];  // buckets longest sentence first, the invalid bucket last
  int keyv[kGroupMaxS + 1];   // sort key of each bucket
  int keyc[kMaxTpad + 2];     // buckets per key, then the key's write cursor
  int wsum[2][16];
};

// The grouping of one batch by the 1024 threads of a block.
__device__ void group_rows_block(int B, int S, int G, const int32_t* __restrict__ sent_id,
                                 const int32_t* __restrict__ len, int Tpad, int32_t* __restrict__ perm,
                                 int4* __restrict__ tiles, int32_t* __restrict__ n_tiles, GroupScratch& sh) {
  int* cnt = sh.cnt;
  int* order = sh.order;
  int* keyv = sh.keyv;
  int* keyc = sh.keyc;
  auto& wsum = sh.wsum;
  const int tid = threadIdx.x, NB = S + 1, NK = Tpad + 1;
  // The first kGroupRowsHeld rows per thread keep their bucket in registers
  // from the count to the scatter, and every id and length is loaded before
  // any is used, so the block waits for one round trip to memory, not one per
  // row.  Rows past the first 1024 x kGroupRowsHeld are read again.
  constexpr int RH = kGroupRowsHeld;
  int bk[RH];
#pragma unroll
  for (int r = 0; r < RH; ++r) {
    const int b = tid + 1024 * r;
    bk[r] = b < B ? sent_id[b] : 0;
  }
  const int l0 = tid < S ? len[tid] : 0;
  for (int i = tid; i < NB; i += 1024) cnt[i] = 0;
  for (int k = tid; k < NK; k += 1024) keyc[k] = 0;
  __syncthreads();
  // rows per bucket, and the key of each bucket: Tpad - length (0 for the
  // longest sentence); the invalid bucket sorts last
#pragma unroll
  for (int r = 0; r < RH; ++r) {
    const int b = tid + 1024 * r, s = bk[r];
    bk[r] = (s >= 0 && s < S) ? s : S;
    if (b < B) atomicAdd(&cnt[bk[r]], 1);
  }
  for (int b = tid + 1024 * RH; b < B; b += 1024) {
    const int s = sent_id[b];
    atomicAdd(&cnt[(s >= 0 && s < S) ? s : S], 1);
  }
  for (int i = tid; i < NB; i += 1024) {
    const int li = i == tid ? l0 : (i < S ? len[i] : 0);
    const int k = i < S ? Tpad - min(max(li, 0), Tpad) : Tpad;
    keyv[i] = k;
    atomicAdd(&keyc[k], 1);
  }
  __syncthreads();
  // exclusive scan of the key counts (NK <= 1025: thread t owns keys [2t, 2t+2))
  {
    const int k0 = 2 * tid, k1 = k0 + 1;
    const int c0 = k0 < NK ? keyc[k0] : 0, c1 = k1 < NK ? keyc[k1] : 0;
    int base = c0 + c1, unused = 0;
    block_scan2(base, unused, wsum);
    if (k0 < NK) keyc[k0] = base;
    if (k1 < NK) keyc[k1] = base + c0;
    __syncthreads();
  }
  for (int i = tid; i < NB; i += 1024) order[atomicAdd(&keyc[keyv[i]], 1)] = i;
  __syncthreads();
  // exclusive scans of the row and tile counts in that order; thread tid owns ranks [lo, hi)
  const int per = (NB + 1023) / 1024, lo = tid * per < NB ? tid * per : NB, hi = lo + per < NB ? lo + per : NB;
  int rs = 0, ts = 0;
  for (int j = lo; j < hi; ++j) {
    const int n = cnt[order[j]];
    rs += n;
    ts += (n + G - 1) / G;
  }
  int roff = rs, toff = ts;
  const int2 tot = block_scan2(roff, toff, wsum);
  if (tid == 0) *n_tiles = tot.y;
  for (int j = lo; j < hi; ++j) {
    const int i = order[j], n = cnt[i];
    for (int k = 0; k * G < n; ++k) tiles[toff + k] = make_int4(i < S ? i : -1, roff + k * G, min(G, n - k * G), 0);
    toff += (n + G - 1) / G;
    cnt[i] = roff;  // becomes the bucket's write cursor
    roff += n;
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < RH; ++r) {
    const int b = tid + 1024 * r;
    if (b < B) perm[atomicAdd(&cnt[bk[r]], 1)] = b;
  }
  for (int b = tid + 1024 * RH; b < B; b += 1024) {
    const int s = sent_id[b];
    perm[atomicAdd(&cnt[(s >= 0 && s < S) ? s : S], 1)] = b;
  }
}

__global__ __launch_bounds__(1024) void k_group_rows(int B, int S, int G, const int32_t* __restrict__ sent_id,
                                                     const int32_t* __restrict__ len, int Tpad,
                                                     int32_t* __restrict__ perm, int4* __restrict__ tiles,
                                                     int32_t* __restrict__ n_tiles) {
  __shared__ GroupScratch sh;
  group_rows_block(B, S, G, sent_id, len, Tpad, perm, tiles, n_tiles, sh);
}

struct GroupLevels {
  GroupLevel l[kMaxGroupLevels];
};

// Block b groups batch b of the launch.
__global__ __launch_bounds__(1024) void k_group_levels(GroupLevels lv, int S, const int32_t* __restrict__ len,
                                                       int Tpad) {
  __shared__ GroupScratch sh;
  const GroupLevel& g = lv.l[blockIdx.x];
  group_rows_block(g.B, S, g.G, g.sent_id, len, Tpad, g.grp.perm, g.grp.tiles, g.grp.n_tiles, sh);
}

hipError_t launch_group_levels(const GroupLevel* lv, int n, int S, const int32_t* len, int Tpad, hipStream_t st) {
  if (S > kGroupMaxS || Tpad > kMaxTpad) return hipErrorInvalidValue;
  for (int i0 = 0; i0 < n; i0 += kMaxGroupLevels) {
    GroupLevels g{};
    const int k = std::min(kMaxGroupLevels, n - i0);
    for (int i = 0; i < k; ++i) g.l[i] = lv[i0 + i];
    hipLaunchKernelGGL(k_group_levels, dim3(k), dim3(1024), 0, st, g, S, len, Tpad);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

int attn_rows_per_tile(int B, int cus) {
  int G = kAttnGroup;
  while (G > 1 && 2 * ceil_div(B, G) < cus) G /= 2;
  return G;
}

// Cross-lane exchanges of gfx950 for the wave sums below.  swap32(x, y)
// returns [x's two 32-lane halves added | y's halves added]: one
// v_permlane32_swap trades x's upper half for y's lower half.  swap16 does
// the same for the rows of 16 lanes: [x0 + x1, y0 + y1, x2 + x3, y2 + y3] for
// rows x0..x3 and y0..y3.  (The pair's elements are read into scalars before
// any bit cast: a bit cast of an element of the returned vector read
// element 0 for both.)
__device__ __forceinline__ float swap32_add(float x, float y) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, x), __builtin_bit_cast(unsigned, y),
                                                  false, false);
  const unsigned a = r[0], b = r[1];
  return __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
}
__device__ __forceinline__ float swap16_add(float x, float y) {
  const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(unsigned, x), __builtin_bit_cast(unsigned, y),
                                                  false, false);
  const unsigned a = r[0], b = r[1];
  return __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
}
// x plus the value of the lane n places higher in its row of 16 (0 past the
// row's end): a DPP row shift.
template <int N>
__device__ __forceinline__ float add_row_shl(float x) {
  const int y = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x100 + N, 0xf, 0xf, false);
  return x + __builtin_bit_cast(float, y);
}

// Sums of G values (G = 1, 2 or 4) over the 64 lanes of a wave: the sum of
// v[g] ends in lane g * (64 / G).  Two halving exchanges (32 lanes, then
// 16) each add two values per exchange, then four DPP shifts sum each row
// of 16 lanes into its first lane: seven cross-lane operations with no
// selects, where a butterfly over lane-chosen array elements compiled to
// chains of compares and selects around seven LDS permutes.
template <int G>
__device__ __forceinline__ float wave_sums(float (&v)[G]) {
  static_assert(G == 1 || G == 2 || G == 4, "one, two or four values per lane");
  float w;
  if constexpr (G == 4) {
    w = swap16_add(swap32_add(v[0], v[2]), swap32_add(v[1], v[3]));  // rows 0..3 in 16-lane rows 0..3
  } else {
    const float h = swap32_add(v[0], v[G - 1]);  // G = 2: [v0 | v1]; G = 1: both halves v0
    w = swap16_add(h, h);
  }
  w = add_row_shl<1>(w);
  w = add_row_shl<2>(w);
  w = add_row_shl<4>(w);
  return add_row_shl<8>(w);
}

template <int G, int NQ, int NW>
__device__ __forceinline__ void attention_tile(const int4 tl, int A, int C, int Tpad, QuerySrc q,
                                               const float* __restrict__ kfac, const float* __restrict__ pctx,
                                               const int32_t* __restrict__ kbig, const float* __restrict__ ctx,
                                               const int32_t* __restrict__ len, const int32_t* __restrict__ perm,
                                               const float* __restrict__ v, float* __restrict__ c,
                                               float* __restrict__ alpha, f32x4* qs, float* e, int* rows, int wave,
                                               int lane, int A4, int C4, int c_bf16, int npg) {
  constexpr int NT = NW * 64;
  const int s = tl.x, n = tl.z;
  if (threadIdx.x < G) rows[threadIdx.x] = (int)threadIdx.x < n ? (perm ? perm[tl.y + threadIdx.x] : tl.y + (int)threadIdx.x) : 0;
  __syncthreads();
  if (s < 0) {  // rows with an invalid sentence: flagged and NaN-ed by the combine kernel
    for (int g = 0; g < n; ++g) {
      for (int k4 = threadIdx.x; k4 < C4; k4 += NT) store_c4(c, (int64_t)rows[g] * C + 4 * k4, zero4(), c_bf16);
      if (alpha)
        for (int i = threadIdx.x; i < Tpad; i += NT) alpha[(int64_t)rows[g] * Tpad + i] = 0.f;
    }
    return;
  }
  // query factors 2^{c q} in LDS and weights -2 v in registers (see score_term);
  // rows past the tile's count get factor 0 and are dropped
  bool big = false;
  for (int idx = threadIdx.x; idx < G * A4; idx += NT) {
    const int g = idx / A4, a4 = idx - g * A4;
    const f32x4 qv = g < n ? load_q(q, rows[g], A, a4) : zero4();
    big |= factor_big(qv);
    qs[idx] = g < n ? tanh_factor(qv) : zero4();
  }
  f32x4 vv[NQ];
#pragma unroll
  for (int k = 0; k < NQ; ++k) {
    const int a4 = lane + 64 * k;
    vv[k] = a4 < A4 ? *(const f32x4*)(v + 4 * a4) * -2.f : zero4();
  }
  const bool exact = __syncthreads_or(big) && kbig[s];
  const int L = len[s];
  // Tiles of fewer than 4 rows come from batches that leave the CUs short of
  // tiles, where a tile's latency sets the kernel's: a wave then loads the
  // keys of U positions (16 vectors a lane) before scoring any of them.
  constexpr int U = G < 4 ? (16 / NQ < 4 ? 16 / NQ : 4) : 1;
  auto score = [&](auto exact_tag, const float* P) {
    constexpr bool EX = decltype(exact_tag)::value;
    for (int i0 = wave; i0 < L; i0 += NW * U) {
      f32x4 p[U][NQ];
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int k = 0; k < NQ; ++k) {
          const int i = i0 + u * NW, a4 = lane + 64 * k;
          p[u][k] = (i < L && a4 < A4) ? *(const f32x4*)(P + (int64_t)i * A + 4 * a4) : zero4();
        }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u * NW;
        if (i >= L) break;  // uniform over the wave
        float acc[G];
#pragma unroll
        for (int g = 0; g < G; ++g) acc[g] = 0.f;
#pragma unroll
        for (int k = 0; k < NQ; ++k) {
          const int a4 = lane + 64 * k;
          if (a4 < A4) {
#pragma unroll
            for (int g = 0; g < G; ++g) {
              const f32x4 qq = qs[g * A4 + a4];
#pragma unroll
              for (int x = 0; x < 4; ++x) acc[g] = score_term_t<EX>(p[u][k][x], qq[x], vv[k][x], acc[g]);
            }
          }
        }
        const float r = wave_sums<G>(acc);
        if ((lane & (64 / G - 1)) == 0) e[(lane / (64 / G)) * Tpad + i] = r;
      }
    }
  };
  if (exact) {  // the queries themselves replace their factors (see kFactorSafe)
    for (int idx = threadIdx.x; idx < G * A4; idx += NT) {
      const int g = idx / A4, a4 = idx - g * A4;
      qs[idx] = g < n ? load_q(q, rows[g], A, a4) : zero4();
    }
    __syncthreads();
    score(std::true_type{}, pctx + (int64_t)s * Tpad * A);
  } else {
    score(std::false_type{}, kfac + (int64_t)s * Tpad * A);
  }
  __syncthreads();
  for (int g = wave; g < n; g += NW) {
    float* eg = e + g * Tpad;
    float mx = -INFINITY;
    for (int i = lane; i < L; i += 64) mx = fmaxf(mx, eg[i]);
    mx = wave_max(mx);
    float sum = 0.f;
    for (int i = lane; i < L; i += 64) sum += expf(eg[i] - mx);
    const float inv = 1.f / wave_sum(sum);
    for (int i = lane; i < L; i += 64) eg[i] = expf(eg[i] - mx) * inv;
    if (alpha)
      for (int i = lane; i < Tpad; i += 64) alpha[(int64_t)rows[g] * Tpad + i] = i < L ? eg[i] : 0.f;
  }
  __syncthreads();
  // Context.  With more threads than float4 columns (npg > 1), the threads
  // of position group pg take the column k4 = tid % C4 over the pg-th of npg
  // contiguous ranges of positions, and group 0 adds the other groups'
  // partial sums (left in LDS over the queries, dead by now) in group order:
  // each thread then waits for a fraction of the annotations' round trips.
  const f32x4* X = (const f32x4*)(ctx + (int64_t)s * Tpad * C);
  const int pg = npg > 1 ? (int)threadIdx.x / C4 : 0;
  const int i_lo = npg > 1 ? L * pg / npg : 0, i_hi = npg > 1 ? L * (pg + 1) / npg : L;
  const int k_first = npg > 1 ? (int)threadIdx.x - pg * C4 : (int)threadIdx.x;
  for (int k4 = k_first; k4 < C4 && pg < npg; k4 += (npg > 1 ? C4 : NT)) {
    f32x4 acc[G];
#pragma unroll
    for (int g = 0; g < G; ++g) acc[g] = zero4();
    auto add = [&](const f32x4& x, int i) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float a = e[g * Tpad + i];
        acc[g][0] += a * x[0];
        acc[g][1] += a * x[1];
        acc[g][2] += a * x[2];
        acc[g][3] += a * x[3];
      }
    };
    // NMT_ATTN_CU annotations are loaded before any is used, so that many
    // loads are in flight per wave instead of one or two (each round trip to
    // L2 or beyond is otherwise paid once per position); the sums still run
    // over the positions in order.
    // Tiles of fewer rows hold fewer accumulators and keep twice the loads
    // in flight.
    constexpr int CU = G >= 4 ? NMT_ATTN_CU : 2 * NMT_ATTN_CU;
    int i = i_lo;
    for (; i + CU <= i_hi; i += CU) {
      f32x4 x[CU];
#pragma unroll
      for (int u = 0; u < CU; ++u) x[u] = X[(int64_t)(i + u) * C4 + k4];
#pragma unroll
      for (int u = 0; u < CU; ++u) add(x[u], i + u);
    }
    for (; i < i_hi; ++i) add(X[(int64_t)i * C4 + k4], i);
    if (npg > 1) {
      if (pg > 0) {
#pragma unroll
        for (int g = 0; g < G; ++g) qs[((pg - 1) * G + g) * C4 + k4] = acc[g];
      }
      __syncthreads();
      if (pg == 0) {
        for (int q = 1; q < npg; ++q)
#pragma unroll
          for (int g = 0; g < G; ++g) acc[g] += qs[((q - 1) * G + g) * C4 + k4];
      }
    }
    if (pg == 0) {
#pragma unroll
      for (int g = 0; g < G; ++g)
        if (g < n) store_c4(c, (int64_t)rows[g] * C + 4 * k4, acc[g], c_bf16);
    }
  }
  if (npg > 1 && (int)threadIdx.x >= npg * C4) __syncthreads();  // threads without a column still meet the barrier
}

// One block (NW waves) per tile of up to G rows of one sentence.  The rows'
// queries sit in LDS; wave w takes source positions w, w+NW, ..., loads the
// position's key once and scores it against all G rows at once (rows past
// the tile's count score zero queries and are dropped), each lane covering
// float4 pieces of the attention width; then one wave per row normalises the
// scores; finally every thread accumulates a float4 piece of the context of
// all rows, reading each annotation once.
template <int G, int NQ, int NW>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(NQ <= 4 ? (G < 4 ? 4 : 8) : 1))) void
k_attention_grouped(
    int A, int C, int Tpad, QuerySrc q, const float* __restrict__ kfac, const float* __restrict__ pctx,
    const int32_t* __restrict__ kbig, const float* __restrict__ ctx, const int32_t* __restrict__ len,
    const int32_t* __restrict__ perm, const int4* __restrict__ tiles,
    const int32_t* __restrict__ n_tiles, const float* __restrict__ v, float* __restrict__ c,
    float* __restrict__ alpha, int c_bf16, int round, int npg, int one_s, int one_sentence_B) {
  // queries [G][A/4] (later the context's partial sums [npg-1][G][C/4]), then scores [G][Tpad]
  extern __shared__ f32x4 dyn[];
  __shared__ int rows[G];
  // one_sentence_B > 0: a batch of that many rows, all of sentence one_s,
  // tiled in row order with no grouping kernel (every tile the same length)
  const int nt = one_sentence_B > 0 ? (one_sentence_B + G - 1) / G : *n_tiles;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int A4 = A / 4, C4 = C / 4;
  f32x4* qs = dyn;
  float* e = (float*)(dyn + max(G * A4, (npg - 1) * G * C4));
  int t = blockIdx.x;
  if (t >= nt) return;
  // Blocks are handed to the CUs in order, one per CU per round of `round`
  // blocks, and the tiles come longest first.  Every other round takes its
  // tiles in reverse, so the CU that got the longest tile of one round gets
  // the shortest of the next, and the CUs' total lengths even out.
  if (round > 0 && one_sentence_B == 0) {
    const int r = t / round, p = t - r * round;
    if (r & 1) t = r * round + (min(round, nt - r * round) - 1 - p);
  }
  const int4 tl = one_sentence_B > 0 ? make_int4(one_s, t * G, min(G, one_sentence_B - t * G), 0) : tiles[t];
  attention_tile<G, NQ, NW>(tl, A, C, Tpad, q, kfac, pctx, kbig, ctx, len, one_sentence_B > 0 ? nullptr : perm, v, c,
                            alpha, qs, e, rows, wave, lane, A4, C4, c_bf16, npg);
}

template <int G, int NQ>
static void attention_grouped(int B, int A, int C, int Tpad, QuerySrc q, const float* kfac, const float* pctx,
                              const int32_t* kbig, const float* ctx, const int32_t* len, const AttnGroups& grp, int S, const float* v, float* c,
                              float* alpha, int c_bf16, int cus, hipStream_t st, int one_s) {
  // at least the number of tiles (exactly, for one sentence)
  const int grid = one_s >= 0 ? ceil_div(B, G) : (int)std::min<int64_t>(B, (int64_t)ceil_div(B, G) + S + 1);
  const int one_B = one_s >= 0 ? B : 0;
  const int round = NMT_ATTN_SNAKE ? cus : 0;
  // Position groups of the context phase: whole waves per group (C/4 a
  // multiple of 64), so every wave meets its one barrier.
  const int C4 = C / 4;
  auto groups = [&](int nt) { return (C4 % 64 == 0 && nt >= 2 * C4) ? nt / C4 : 1; };
  auto lds_bytes = [&](int npg) {
    return (size_t)std::max(G * (A / 4), (npg - 1) * G * C4) * 16 + (size_t)G * Tpad * 4;
  };
  // Few tiles (about two per CU or fewer, e.g. 2,000 rows in 20 sentences)
  // leave the CUs short of waves to hide memory latency with: twice the
  // waves per tile then take half the positions each (fp32 enru_b2000
  // 41.9 -> 36.1 us).  With four tiles per CU (4,096 rows) 8 waves measured
  // faster (70.6 against 75.1 us).
  if (grid <= kAttnWideTiles) {
    const int npg = groups(2 * kAttnWaves * 64);
    hipLaunchKernelGGL((k_attention_grouped<G, NQ, 2 * kAttnWaves>), dim3(grid), dim3(2 * kAttnWaves * 64),
                       lds_bytes(npg), st, A, C, Tpad, q, kfac, pctx, kbig, ctx, len, grp.perm, grp.tiles, grp.n_tiles,
                       v, c, alpha, c_bf16, round, npg, one_s, one_B);
  } else {
    const int npg = groups(kAttnWaves * 64);
    hipLaunchKernelGGL((k_attention_grouped<G, NQ, kAttnWaves>), dim3(grid), dim3(kAttnWaves * 64), lds_bytes(npg), st,
                       A, C, Tpad, q, kfac, pctx, kbig, ctx, len, grp.perm, grp.tiles, grp.n_tiles, v, c, alpha, c_bf16,
                       round, npg, one_s, one_B);
  }
}

template <int NQ>
static void attention_nq(int B, int A, int C, int Tpad, QuerySrc q, const float* kfac, const float* pctx,
                         const int32_t* kbig, const float* ctx, const int32_t* len, const int32_t* sent_id, const AttnGroups& grp, int S, const float* v,
                         float* c, float* alpha, int c_bf16, int cus, hipStream_t st, bool grouped) {
  if (S > kGroupMaxS || !grp.perm) {
    hipLaunchKernelGGL(k_attention<NQ>, dim3(B), dim3(256), 0, st, B, A, C, Tpad, q, kfac, pctx, kbig, ctx, len,
                       sent_id, S, v, c, alpha, c_bf16);
    return;
  }
  // Rows per tile: 4, so that a block reads each key and annotation once for
  // four rows.  A tile runs on one CU, so with few tiles the longest
  // sentence's tile sets the kernel's duration (about 26 us for 80 positions,
  // whatever the batch): batches that would give fewer tiles than half the
  // CUs take tiles of 2 rows, or 1, spreading the same work over more CUs.
  // (At 1,000 rows of one sentence, 2-row tiles measured slower, 32 -> 40 us:
  // twice the tiles read the one sentence's keys at once.)
  const int G = attn_rows_per_tile(B, cus);
  // Rows of a single sentence need no grouping: their tiles are runs of
  // consecutive rows.  That holds for a source of one sentence (a row with
  // another sentence id is still flagged, and its log p made NaN, by the
  // combine; its attention then reads sentence 0), or when the caller knows
  // every row's sentence (grp.one_sentence, checked against S on the host).
  const int one = grp.one_sentence >= 0 ? grp.one_sentence : (!grouped && S == 1 ? 0 : -1);
  if (!grouped && one < 0)
    hipLaunchKernelGGL(k_group_rows, dim3(1), dim3(1024), 0, st, B, S, G, sent_id, len, Tpad, grp.perm, grp.tiles,
                       grp.n_tiles);
  if (G >= 4)
    attention_grouped<4, NQ>(B, A, C, Tpad, q, kfac, pctx, kbig, ctx, len, grp, S, v, c, alpha, c_bf16, cus, st, one);
  else if (G == 2)
    attention_grouped<2, NQ>(B, A, C, Tpad, q, kfac, pctx, kbig, ctx, len, grp, S, v, c, alpha, c_bf16, cus, st, one);
  else
    attention_grouped<1, NQ>(B, A, C, Tpad, q, kfac, pctx, kbig, ctx, len, grp, S, v, c, alpha, c_bf16, cus, st, one);
}

hipError_t launch_attention(int B, int A, int C, int Tpad, QuerySrc q, const float* kfac, const float* pctx,
                            const int32_t* kbig, const float* ctx, const int32_t* len, const int32_t* sent_id, int S, const float* v, float* c, float* alpha,
                            const AttnGroups& grp, bool c_bf16, int cus, hipStream_t st, bool grouped) {
  if (B <= 0) return hipSuccess;
  const int nq = ceil_div(A, 256);
  if (nq <= 1)
    attention_nq<1>(B, A, C, Tpad, q, kfac, pctx, kbig, ctx, len, sent_id, grp, S, v, c, alpha, c_bf16 ? 1 : 0, cus, st, grouped);
  else if (nq <= 2)
    attention_nq<2>(B, A, C, Tpad, q, kfac, pctx, kbig, ctx, len, sent_id, grp, S, v, c, alpha, c_bf16 ? 1 : 0, cus, st, grouped);
  else if (nq <= 4)
    attention_nq<4>(B, A, C, Tpad, q, kfac, pctx, kbig, ctx, len, sent_id, grp, S, v, c, alpha, c_bf16 ? 1 : 0, cus, st, grouped);
  else if (nq <= 8)
    attention_nq<8>(B, A, C, Tpad, q, kfac, pctx, kbig, ctx, len, sent_id, grp, S, v, c, alpha, c_bf16 ? 1 : 0, cus, st, grouped);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// Widens a bf16 matrix [rows x cols] with row stride ld to a dense fp32 one
// (bf16 intermediates for the debug outputs).
__global__ void k_bf16_to_f32(int64_t rows, int cols, int64_t ld, const __bf16* __restrict__ x,
                              float* __restrict__ y) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < rows * cols) y[i] = (float)x[(i / cols) * ld + i % cols];
}

hipError_t launch_bf16_to_f32(const void* x, int64_t rows, int cols, int64_t ld, float* y, hipStream_t st) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  const int64_t n = rows * cols;
  hipLaunchKernelGGL(k_bf16_to_f32, dim3((unsigned)ceil_div(n, (int64_t)256)), dim3(256), 0, st, rows, cols, ld,
                     (const __bf16*)x, y);
  return hipGetLastError();
}

// ------------------------------------------------------ source helpers

__global__ void k_check_src_ids(int S, int Tpad, const int32_t* ids, const int32_t* len, int V_src, int* err) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)S * Tpad) return;
  const int s = (int)(i / Tpad), p = (int)(i % Tpad);
  if (p < len[s] && (ids[i] < 0 || ids[i] >= V_src)) atomicOr(err, 1);
}

hipError_t launch_check_src_ids(int S, int Tpad, const int32_t* ids, const int32_t* len, int V_src, int* err,
                                hipStream_t st) {
  const int64_t n = (int64_t)S * Tpad;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_check_src_ids, dim3(ceil_div(n, 256)), dim3(256), 0, st, S, Tpad, ids, len, V_src, err);
  return hipGetLastError();
}

__global__ void k_masked_copy(int S, int Tpad, int C, const float* src, const int32_t* len, float* dst) {
  const int64_t i4 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int C4 = C / 4;
  if (i4 >= (int64_t)S * Tpad * C4) return;
  const int64_t pos = i4 / C4;
  const int s = (int)(pos / Tpad), p = (int)(pos % Tpad);
  ((f32x4*)dst)[i4] = p < len[s] ? ((const f32x4*)src)[i4] : zero4();
}

hipError_t launch_masked_copy(int S, int Tpad, int C, const float* src, const int32_t* len, float* dst,
                              hipStream_t st) {
  const int64_t n = (int64_t)S * Tpad * (C / 4);
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_masked_copy, dim3(ceil_div(n, 256)), dim3(256), 0, st, S, Tpad, C, src, len, dst);
  return hipGetLastError();
}

// mean over the unmasked positions of each sentence: one block per sentence.
__global__ void k_masked_mean(int Tpad, int C, const float* ctx, const int32_t* len, float* mean) {
  const int s = blockIdx.x, L = len[s];
  const float* X = ctx + (int64_t)s * Tpad * C;
  for (int k = threadIdx.x; k < C; k += blockDim.x) {
    float acc = 0.f;
    for (int i = 0; i < L; ++i) acc += X[(int64_t)i * C + k];
    mean[(int64_t)s * C + k] = acc / (float)L;
  }
}

hipError_t launch_masked_mean(int S, int Tpad, int C, const float* ctx, const int32_t* len, float* mean,
                              hipStream_t st) {
  if (S <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_masked_mean, dim3(S), dim3(256), 0, st, Tpad, C, ctx, len, mean);
  return hipGetLastError();
}

// ------------------------------------------------- several models

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
// Nearest bf16, ties to even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// One parameter buffer of the weighted model average: element i is
// sum_k coef[k] * src[k][i], accumulated in fp32 in model order with fused
// multiply-adds, then stored in the buffer's type (bf16 nearest-even; fp32,
// or fp32 rounded to a bf16 value when the model keeps bf16 parameters).
// The model loop is unrolled to the table size so the table stays in
// registers.
__global__ void k_average(int K, int64_t n, ModelTable tab, int kind, int round_bf16, void* __restrict__ dst) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    float acc = 0.f;
#pragma unroll
    for (int k = 0; k < kMaxModels; ++k)
      if (k < K) {
        const float x = kind == 2 ? bf16_bits_to_f32(((const uint16_t*)tab.p[k])[i]) : ((const float*)tab.p[k])[i];
        acc = fmaf(tab.w[k], x, acc);
      }
    if (kind == 2)
      ((uint16_t*)dst)[i] = f32_to_bf16_bits(acc);
    else
      ((float*)dst)[i] = round_bf16 ? bf16_bits_to_f32(f32_to_bf16_bits(acc)) : acc;
  }
}

hipError_t launch_average(int K, int64_t n, const ModelTable& tab, int kind, bool round_bf16, void* dst,
                          hipStream_t st) {
  if (K < 1 || K > kMaxModels || (kind != 1 && kind != 2)) return hipErrorInvalidValue;
  if (n <= 0) return hipSuccess;
  const int64_t blocks = ceil_div(n, 256) < 8192 ? ceil_div(n, 256) : 8192;
  hipLaunchKernelGGL(k_average, dim3((unsigned)blocks), dim3(256), 0, st, K, n, tab, kind, round_bf16 ? 1 : 0, dst);
  return hipGetLastError();
}

// out[b] = sum_k w[k] * logp[k*B + b], in model order.
__global__ void k_weighted_sum(int K, int B, const float* __restrict__ logp, ModelTable tab, float* __restrict__ out) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  float acc = 0.f;
#pragma unroll
  for (int k = 0; k < kMaxModels; ++k)
    if (k < K) acc = fmaf(tab.w[k], logp[(int64_t)k * B + b], acc);
  out[b] = acc;
}

hipError_t launch_weighted_sum(int K, int B, const float* logp, const ModelTable& tab, float* out, hipStream_t st) {
  if (K < 1 || K > kMaxModels) return hipErrorInvalidValue;
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_weighted_sum, dim3(ceil_div(B, 256)), dim3(256), 0, st, K, B, logp, tab, out);
  return hipGetLastError();
}

}  // namespace nmt
