// HIP kernels of the ETA decode path for gfx950 (CDNA4, wave64).
//
// Kernels and what they compute (paper: "Elastic Threshold Attention: Learned
// Contextual Sparsity for Long-Context Decoding"):
//   summaries_kernel  mu, sigma, M of every full KV block   (Sec. "Block-Based Scanning via
//                                                            Dual Metadata Caching")
//   predict_kernel    tau = concat(q) W + bias                (Eq. tau_pred)
//   screen_kernel     Score_dual per block and head, threshold, pins, top-1 rescue,
//                     GQA union and its compaction           (Eq. dual_bound_eq; Alg.
//                                                            "Hardware-Aligned Block-Sparse
//                                                            Decoding (Inference)")
//   split_kernel      gated online softmax over a slice of the union list plus the
//                     tail; one (max, sum, acc) partial per head and split
//                                                           (Eq. mult_attn; App. "Chunked
//                                                            Decoding and Two-Stage Reduction")
//   combine_kernel    log-sum-exp merge of the partials      (same appendix)
//   calib_kernel,     offline calibration histogram and bisection
//   calib_solve_kernel                                       (Alg. "calibration")
// The gated prefill forward is in eta_prefill.hip.  The dense baseline reuses split_kernel / combine_kernel with every block and
// no gate.
//
// All arithmetic is fp32 (bf16 inputs are widened exactly); reductions use a
// fixed order, so results are bitwise reproducible.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>

#include "eta_device.h"
#include "eta_index.h"
#include "eta_internal.h"

// The source compiles to three objects, in parallel (ETA_PART): 0 holds every
// kernel but split decode, and the host launchers; 1 and 2 hold split decode
// on bf16 and fp32 caches.
#ifndef ETA_PART
#define ETA_PART 0
#endif

namespace eta {
namespace {

__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ uint16_t to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// fp32 -> 8-bit E4M3 code (bias 7, 3 fraction bits), round to nearest even;
// magnitudes from 464 (the tie past 448, the largest finite value) saturate
// to 448, NaN gives the NaN code.
__device__ __forceinline__ uint8_t to_e4m3(float f) {
  const uint32_t sgn = (__float_as_uint(f) >> 24) & 0x80u;
  const float a = fabsf(f);
  if (!(a == a)) return (uint8_t)(sgn | 0x7fu);
  if (a >= 464.0f) return (uint8_t)(sgn | 0x7eu);
  if (a < 0.015625f)                              // below 2^-6: multiples of 2^-9
    return (uint8_t)(sgn | (uint32_t)rintf(a * 512.0f));   // 0 .. 8 (8: the code of 2^-6)
  const uint32_t au = __float_as_uint(a);
  int e = (int)(au >> 23) - 127;                  // -6 .. 8
  uint32_t keep = (au >> 20) & 7u;
  const uint32_t rest = au & 0xfffffu;
  if (rest > 0x80000u || (rest == 0x80000u && (keep & 1u))) ++keep;
  if (keep == 8u) {
    keep = 0u;
    ++e;
  }
  return (uint8_t)(sgn | ((uint32_t)(e + 7) << 3) | keep);
}

// record element -> fp32 (E4M3 codes decoded exactly by the hardware conversion)
__device__ __forceinline__ float stat_f32(float x) { return x; }
__device__ __forceinline__ float stat_f32(_Float16 x) { return (float)x; }
__device__ __forceinline__ float stat_f32(uint8_t x) {
  return __builtin_amdgcn_cvt_f32_fp8((int)x, 0);
}

// Four consecutive records of one coordinate row (one 16-, 8- or 4-byte load),
// and their fp32 values (the same conversions as stat_f32).
template <typename ST>
struct alignas(4 * sizeof(ST)) Rec4 {
  ST v[4];
};
template <typename ST>
__device__ __forceinline__ void rec4_f32(const Rec4<ST>& r, float (&f)[4]) {
  if constexpr (sizeof(ST) == 1) {
    const int word = (int)__builtin_bit_cast(uint32_t, r);
    f[0] = __builtin_amdgcn_cvt_f32_fp8(word, 0);
    f[1] = __builtin_amdgcn_cvt_f32_fp8(word, 1);
    f[2] = __builtin_amdgcn_cvt_f32_fp8(word, 2);
    f[3] = __builtin_amdgcn_cvt_f32_fp8(word, 3);
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) f[e] = stat_f32(r.v[e]);
  }
}

// Element access for the two storage types: float and bf16 (raw uint16 bits).
template <typename T>
struct Elem;

template <>
struct Elem<float> {
  static __device__ __forceinline__ float get(const float* p, int64_t i) { return p[i]; }
  static __device__ __forceinline__ void load8(const float* p, float (&x)[8]) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
  }
  template <int N>
  static __device__ __forceinline__ void loadn(const float* p, float (&x)[N]) {
    if constexpr (N == 1) {
      x[0] = *p;
    } else {
      const float2 a = *reinterpret_cast<const float2*>(p);
      x[0] = a.x; x[1] = a.y;
    }
  }
};

template <>
struct Elem<uint16_t> {
  static __device__ __forceinline__ float get(const uint16_t* p, int64_t i) { return bf16lo(p[i]); }
  static __device__ __forceinline__ void load8(const uint16_t* p, float (&x)[8]) {
    const uint4 a = *reinterpret_cast<const uint4*>(p);
    x[0] = bf16lo(a.x); x[1] = bf16hi(a.x); x[2] = bf16lo(a.y); x[3] = bf16hi(a.y);
    x[4] = bf16lo(a.z); x[5] = bf16hi(a.z); x[6] = bf16lo(a.w); x[7] = bf16hi(a.w);
  }
  template <int N>
  static __device__ __forceinline__ void loadn(const uint16_t* p, float (&x)[N]) {
    if constexpr (N == 1) {
      x[0] = bf16lo(*p);
    } else {
      const uint32_t a = *reinterpret_cast<const uint32_t*>(p);
      x[0] = bf16lo(a); x[1] = bf16hi(a);
    }
  }
};

__device__ __forceinline__ float load_q(const void* q, int q_dtype, int64_t idx) {
  if (q_dtype == ETA_DT_F32) return reinterpret_cast<const float*>(q)[idx];
  return bf16lo(reinterpret_cast<const uint16_t*>(q)[idx]);
}

__device__ __forceinline__ void store_out(void* o, int q_dtype, int64_t idx, float x) {
  if (q_dtype == ETA_DT_F32)
    reinterpret_cast<float*>(o)[idx] = x;
  else
    reinterpret_cast<uint16_t*>(o)[idx] = to_bf16(x);
}

// Wavefront-wide butterfly reductions on the vector ALUs (no LDS round trips):
// quad permutes pair lane ^ 1 and lane ^ 2; the 8- and 16-lane mirrors then
// pair lanes holding the same values as lane ^ 4 and lane ^ 8 (all lanes of a
// quad, then of an 8-lane half, are equal by then); the row and half-wave
// swaps hand each lane both operands of lane ^ 16 and lane ^ 32.  Every lane
// ends with the same, bitwise identical result.  Full EXEC only.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}

template <typename Op>
__device__ __forceinline__ float wave_reduce(float x, Op op) {
  x = op(x, dpp_mov<0xB1>(x));    // quad_perm [1,0,3,2]
  x = op(x, dpp_mov<0x4E>(x));    // quad_perm [2,3,0,1]
  x = op(x, dpp_mov<0x141>(x));   // row_half_mirror
  x = op(x, dpp_mov<0x140>(x));   // row_mirror
  const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = op(__uint_as_float(r16[0]), __uint_as_float(r16[1]));
  const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return op(__uint_as_float(r32[0]), __uint_as_float(r32[1]));
}

// (largest value, smallest index among its lanes) over the wavefront, in every
// lane, for N independent pairs: the max / min-index order is a total order, so
// the same steps as wave_reduce pair every lane with every other; the N
// butterflies run stage by stage, interleaved, instead of one after another.
template <int N>
__device__ __forceinline__ void wave_argmax_n(float (&v)[N], int (&i)[N]) {
  auto take = [](float& cv, int& ci, float ov, int oi) {
    if (ov > cv || (ov == cv && oi < ci)) { cv = ov; ci = oi; }
  };
#define ETA_ARGMAX_DPP(CTRL)                                                                    \
  {                                                                                             \
    float ov[N];                                                                                \
    int oi[N];                                                                                  \
    _Pragma("unroll") for (int n = 0; n < N; ++n) {                                             \
      ov[n] = dpp_mov<CTRL>(v[n]);                                                              \
      oi[n] = __float_as_int(dpp_mov<CTRL>(__int_as_float(i[n])));                              \
    }                                                                                           \
    _Pragma("unroll") for (int n = 0; n < N; ++n) take(v[n], i[n], ov[n], oi[n]);               \
  }
  ETA_ARGMAX_DPP(0xB1)
  ETA_ARGMAX_DPP(0x4E)
  ETA_ARGMAX_DPP(0x141)
  ETA_ARGMAX_DPP(0x140)
#undef ETA_ARGMAX_DPP
#pragma unroll
  for (int n = 0; n < N; ++n) {
    const auto rv = __builtin_amdgcn_permlane16_swap(__float_as_uint(v[n]), __float_as_uint(v[n]), false, false);
    const auto ri = __builtin_amdgcn_permlane16_swap((uint32_t)i[n], (uint32_t)i[n], false, false);
    v[n] = __uint_as_float(rv[0]);
    i[n] = (int)ri[0];
    take(v[n], i[n], __uint_as_float(rv[1]), (int)ri[1]);
  }
#pragma unroll
  for (int n = 0; n < N; ++n) {
    const auto rv = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[n]), __float_as_uint(v[n]), false, false);
    const auto ri = __builtin_amdgcn_permlane32_swap((uint32_t)i[n], (uint32_t)i[n], false, false);
    v[n] = __uint_as_float(rv[0]);
    i[n] = (int)ri[0];
    take(v[n], i[n], __uint_as_float(rv[1]), (int)ri[1]);
  }
}

__device__ __forceinline__ float wave_max(float x) {
  return wave_reduce(x, [](float a, float b) { return fmaxf(a, b); });
}
__device__ __forceinline__ float wave_sum(float x) {
  return wave_reduce(x, [](float a, float b) { return a + b; });
}

// Inclusive prefix sum of an integer over the wavefront's lanes, on the vector
// ALUs: shifts by 1, 2, 4 and 8 lanes within each 16-lane row (a lane whose
// source would lie in the previous row adds 0), then each row adds the totals
// of the rows before it, read from lanes 15, 31 and 47.  Lane 63 ends with the
// wavefront's total.  Full EXEC only.
__device__ __forceinline__ int wave_incl_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);   // row_shr:8
  const int r0 = __builtin_amdgcn_readlane(x, 15);
  const int r1 = r0 + __builtin_amdgcn_readlane(x, 31);
  const int r2 = r1 + __builtin_amdgcn_readlane(x, 47);
  const int row = (int)(threadIdx.x & 63) >> 4;
  return x + (row == 0 ? 0 : (row == 1 ? r0 : (row == 2 ? r1 : r2)));
}

// ---------------------------------------------------------------- summaries
//
// One workgroup handles kSumBlocks consecutive full blocks of one (sequence,
// kv head); wavefront w takes blocks w, w + 4, ...  A block is read with
// fully coalesced 16-byte loads: LPR lanes cover one row, so one load covers
// R = 64 / LPR consecutive rows, and lane l keeps the EPL coordinates
// EPL (l % LPR) .. + EPL - 1 of rows l / LPR, l / LPR + R, ...  The block
// stays in registers for the two passes (mean, then mean squared deviation);
// the row norms are summed over the LPR lanes of a row, and the per-lane
// sums over the R row groups.  Results are staged in LDS and written as whole
// rows of kSumBlocks consecutive blocks of the dimension-major output.
//
// Variants: ENV replaces sigma by the sub-block envelope (per coordinate, the
// largest root mean squared deviation from the block mean over contiguous
// sub-blocks of 2^sub_log2 tokens); with prev_lens, the blocks start at
// prev_lens[b] / BS (the blocks completed since then) and at most max_new
// blocks per sequence are written.

constexpr int kSumBlocks = 32;

// Sum over the aligned group of N lanes (N in 8, 16, 32) that holds one row;
// every lane of the group ends with the same value.
template <int N>
__device__ __forceinline__ float lane_group_sum(float x) {
  x += dpp_mov<0xB1>(x);
  x += dpp_mov<0x4E>(x);
  x += dpp_mov<0x141>(x);
  if constexpr (N >= 16) x += dpp_mov<0x140>(x);
  if constexpr (N >= 32) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  return x;
}

// Combines lanes l, l ^ N, l ^ 2N, ... (the same coordinates of the other row
// groups) with op; every lane ends with the combined value.
template <int N, typename Op>
__device__ __forceinline__ float row_group_reduce(float x, Op op) {
  if constexpr (N <= 8) x = op(x, dpp_mov<0x128>(x));   // row_ror:8 = lane ^ 8 in a row
  if constexpr (N <= 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = op(__uint_as_float(r[0]), __uint_as_float(r[1]));
  }
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return op(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Sum over ng (1, 2, 4 or 8) consecutive row groups of N lanes each.
template <int N>
__device__ __forceinline__ float partial_group_sum(float x, int ng) {
  auto swap_sum16 = [](float y) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(y), __float_as_uint(y), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
  };
  auto swap_sum32 = [](float y) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
  };
  if constexpr (N == 8) {
    if (ng >= 2) x += dpp_mov<0x128>(x);
    if (ng >= 4) x = swap_sum16(x);
    if (ng >= 8) x = swap_sum32(x);
  } else if constexpr (N == 16) {
    if (ng >= 2) x = swap_sum16(x);
    if (ng >= 4) x = swap_sum32(x);
  } else {
    if (ng >= 2) x = swap_sum32(x);
  }
  return x;
}

// 16 bytes of K for the summaries: every load covers whole rows (LPR lanes x
// 16 bytes each) read once, so it carries the non-temporal hint (the build over
// 512 MiB of K went from 113 to 99 us with it)
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
template <typename T>
__device__ __forceinline__ uint4 load_nt16(const T* p) {
  return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p)));
}

template <typename KVT>
__device__ __forceinline__ void unpack16(const uint4& u, float (&f)[16 / sizeof(KVT)]) {
  if constexpr (sizeof(KVT) == 2) {
    f[0] = bf16lo(u.x); f[1] = bf16hi(u.x); f[2] = bf16lo(u.y); f[3] = bf16hi(u.y);
    f[4] = bf16lo(u.z); f[5] = bf16hi(u.z); f[6] = bf16lo(u.w); f[7] = bf16hi(u.w);
  } else {
    f[0] = __uint_as_float(u.x); f[1] = __uint_as_float(u.y);
    f[2] = __uint_as_float(u.z); f[3] = __uint_as_float(u.w);
  }
}

template <int D, int BS, typename KVT, bool ENV>
__global__ __launch_bounds__(256) void summaries_kernel(const KVT* __restrict__ k, Geom g,
                                                        const int32_t* __restrict__ seq_lens,
                                                        const int32_t* __restrict__ prev_lens,
                                                        int max_new, int sub_log2,
                                                        void* __restrict__ mu,
                                                        void* __restrict__ sigma,
                                                        float* __restrict__ mx) {
  constexpr int EPL = 16 / (int)sizeof(KVT);   // coordinates per lane and load
  constexpr int LPR = D / EPL;                 // lanes per row
  constexpr int R = 64 / LPR;                  // rows per load
  constexpr int NI = BS / R;                   // loads per lane and block
  constexpr int CH = NI * 4 <= 128 ? NI : 16;  // loads held at once (VGPR budget)
  constexpr int NCH = NI / CH;
  static_assert(LPR >= 8 && LPR <= 32 && NI % CH == 0, "unsupported summary shape");
  // the envelope's sub-block sums over four row groups of 16 lanes (bf16 rows
  // of 128) take the transposed route below when a sub-block spans all four
  constexpr bool TR = ENV && LPR == 16 && EPL == 8;
  const bool tr_on = TR && (1 << sub_log2) >= R;
  __shared__ float mu_s[D][kSumBlocks + 1];
  __shared__ float sg_s[D][kSumBlocks + 1];
  __shared__ float mx_s[kSumBlocks];

  const int gh = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int rg = lane / LPR, cl = lane % LPR;
  const int64_t T = clamp_len(seq_lens, b, g.cap);
  int64_t N = T / BS;
  int64_t j0 = (int64_t)blockIdx.x * kSumBlocks;
  if (prev_lens != nullptr) {
    const int64_t first = clamp_len(prev_lens, b, g.cap) / BS;
    j0 += first;
    if (N > first + max_new) N = first + max_new;
  }
  if (j0 >= N) return;
  const KVT* kb = k + (int64_t)b * g.sb + (int64_t)gh * g.sh;
  const int64_t bg = (int64_t)b * g.Hkv + gh;
  constexpr float inv_bs = 1.0f / BS;

  for (int jj = w; jj < kSumBlocks; jj += 4) {
    const int64_t j = j0 + jj;
    if (j >= N) break;
    const KVT* base = kb + (j * BS + rg) * g.st + cl * EPL;
    uint4 x[CH];
    // all of a chunk's loads are issued before any of them is used
    auto load_chunk = [&](int c) {
#pragma unroll
      for (int i = 0; i < CH; ++i)
        x[i] = load_nt16(base + (int64_t)(R * (c * CH + i)) * g.st);
      __builtin_amdgcn_sched_barrier(0);
    };
    float s[EPL], v[EPL], n2max = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) { s[e] = 0.f; v[e] = 0.f; }
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      load_chunk(c);
#pragma unroll
      for (int i = 0; i < CH; ++i) {
        float f[EPL];
        unpack16<KVT>(x[i], f);
        float n2 = 0.f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) {
          s[e] += f[e];
          n2 = fmaf(f[e], f[e], n2);
        }
        n2max = fmaxf(n2max, lane_group_sum<LPR>(n2));
      }
    }
    float mean[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      mean[e] = row_group_reduce<LPR>(s[e], [](float a, float c) { return a + c; }) * inv_bs;
      s[e] = 0.f;   // pass two keeps the envelope here
    }
    float tr_s[2] = {0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      if constexpr (NCH > 1) {
        load_chunk(c);
      } else {
        // unpack again rather than keep pass one's unpacked values alive
#pragma unroll
        for (int i = 0; i < CH; ++i) asm volatile("" : "+v"(x[i].x), "+v"(x[i].y), "+v"(x[i].z), "+v"(x[i].w));
      }
#pragma unroll
      for (int i = 0; i < CH; ++i) {
        float f[EPL];
        unpack16<KVT>(x[i], f);
#pragma unroll
        for (int e = 0; e < EPL; ++e) {
          const float dv = f[e] - mean[e];
          v[e] = fmaf(dv, dv, v[e]);
        }
        if constexpr (ENV) {
          // a sub-block is ng row groups of kl consecutive loads
          const int sub = 1 << sub_log2;
          const int ng = sub < R ? sub : R, kl = sub > R ? sub / R : 1;
          if (((c * CH + i + 1) & (kl - 1)) == 0) {
            const float inv_sub = 1.0f / (float)sub;
            if (TR && ng == 4) {
              // the eight coordinates' sums over the four row groups at once:
              // each row swap exchanges two coordinates' rows, so the pairwise
              // adds are those of partial_group_sum (same operands, same
              // order) and coordinate 4 m + r ends in row r of tr_s[m]
              float u[4];
#pragma unroll
              for (int p = 0; p < 4; ++p) {
                const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v[2 * p]),
                                                                __float_as_uint(v[2 * p + 1]), false, false);
                u[p] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
              }
#pragma unroll
              for (int m = 0; m < 2; ++m) {
                const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(u[2 * m]),
                                                                __float_as_uint(u[2 * m + 1]), false, false);
                tr_s[m] = fmaxf(tr_s[m], (__uint_as_float(r[0]) + __uint_as_float(r[1])) * inv_sub);
              }
#pragma unroll
              for (int e = 0; e < EPL; ++e) v[e] = 0.f;
            } else {
#pragma unroll
              for (int e = 0; e < EPL; ++e) {
                // the largest mean square deviation; its root is taken once at
                // the end (the root is monotone, so this is the largest root)
                const float t = partial_group_sum<LPR>(v[e], ng);
                s[e] = fmaxf(s[e], t * inv_sub);
                v[e] = 0.f;
              }
            }
          }
        }
      }
    }
    if (TR && tr_on) {
      // row group rg holds coordinates rg and 4 + rg of its lane's eight
      if (rg == 0) {
#pragma unroll
        for (int e = 0; e < EPL; ++e) mu_s[cl * EPL + e][jj] = mean[e];
      }
      sg_s[cl * EPL + rg][jj] = sqrtf(tr_s[0]);
      sg_s[cl * EPL + 4 + rg][jj] = sqrtf(tr_s[1]);
    } else {
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        float sd;
        if constexpr (ENV)
          sd = sqrtf(row_group_reduce<LPR>(s[e], [](float a, float c) { return fmaxf(a, c); }));
        else
          sd = sqrtf(row_group_reduce<LPR>(v[e], [](float a, float c) { return a + c; }) * inv_bs);
        if (rg == 0) {
          mu_s[cl * EPL + e][jj] = mean[e];
          sg_s[cl * EPL + e][jj] = sd;
        }
      }
    }
    n2max = row_group_reduce<LPR>(n2max, [](float a, float c) { return fmaxf(a, c); });
    if (lane == 0) mx_s[jj] = sqrtf(n2max);
  }
  __syncthreads();
  // whole rows of the dimension-major output (blocks j0 .. j0 + nv - 1)
  const int nv = N - j0 < kSumBlocks ? (int)(N - j0) : kSumBlocks;
  const int64_t ob = bg * D * g.ncap + j0;
  const bool f16 = g.stat_dtype == ETA_DT_F16, fp8 = g.stat_dtype == ETA_DT_FP8;
  for (int idx = tid; idx < D * kSumBlocks; idx += 256) {
    const int i = idx / kSumBlocks, jj = idx % kSumBlocks;
    if (jj < nv) {
      const int64_t o = ob + (int64_t)i * g.ncap + jj;
      if (f16) {   // round to nearest even
        reinterpret_cast<_Float16*>(mu)[o] = (_Float16)mu_s[i][jj];
        reinterpret_cast<_Float16*>(sigma)[o] = (_Float16)sg_s[i][jj];
      } else if (fp8) {
        reinterpret_cast<uint8_t*>(mu)[o] = to_e4m3(mu_s[i][jj]);
        reinterpret_cast<uint8_t*>(sigma)[o] = to_e4m3(sg_s[i][jj]);
      } else {
        reinterpret_cast<float*>(mu)[o] = mu_s[i][jj];
        reinterpret_cast<float*>(sigma)[o] = sg_s[i][jj];
      }
    }
  }
  if (tid < nv) mx[bg * g.ncap + j0 + tid] = mx_s[tid];
}

// ---------------------------------------------------------------- predictor
//
// tau[b][h] = sum_j qbar[b][j] W[h][j] + bias[h].  W is head-major: row h holds
// the Hq d weights of head h's threshold (the predictor's (Hq d) x Hq matrix
// transposed), so a workgroup that predicts a few heads reads those heads' rows
// and nothing else.  One fixed summation order is shared by the stand-alone
// predictor and the screening kernel's fused prediction, so both give
// bit-identical thresholds: thread t of a 256-thread workgroup accumulates rows
// j = 1024 p + 4 t + e (passes p = 0, 1, ..., e = 0..3 within each, in that
// order); each wavefront reduces by butterfly; the four wavefront sums are
// added in order; the bias is added last.

constexpr int kPredThreads = 256;
#if ETA_PART == 0
constexpr int kPredCols = 4;                    // heads per stand-alone predictor workgroup
#endif
constexpr int kPredStep = 4 * kPredThreads;     // rows per pass
static_assert(kPredStep == 1024, "pred_row4 (eta_index.h) takes 1024 rows per pass");
// The first kPredPass passes of each thread are loaded into registers by
// pred_load (so a caller can issue them ahead of other loads) and consumed by
// pred_sum, which then continues over any further rows in the same order.
constexpr int kPredPass = 2;

template <int NC>
struct PredRows {
  uint32_t x[kPredPass][4];   // raw query bits (fp32, or bf16 in the low half)
  float w[kPredPass][NC][4];
};

__device__ __forceinline__ float pred_x(uint32_t raw, int q_dtype) {
  return q_dtype == ETA_DT_F32 ? __uint_as_float(raw) : __uint_as_float(raw << 16);
}

// Loads passes p0 .. p0 + kPredPass - 1 of this thread: rows 1024 p + 4 t + e of
// the query and of heads h0 .. h0 + ncols - 1 (ncols <= NC), all unconditional
// (indexes clamped, the unused values zeroed in pred_fma) so that they are in
// flight together; the query is kept as raw bits until pred_fma so that no
// conversion waits for its load.  VEC: J a multiple of 4, so each thread's four
// rows are one 8- or 16-byte query load and one 16-byte load per head.
template <int NC, bool VEC>
__device__ __forceinline__ void pred_load(const void* __restrict__ q, int q_dtype, int64_t qoff,
                                          const float* __restrict__ W, int J, int h0, int ncols,
                                          int p0, PredRows<NC>& r) {
#pragma unroll
  for (int p = 0; p < kPredPass; ++p) {
    const int j = (p0 + p) * kPredStep + 4 * (int)threadIdx.x;
    if constexpr (VEC) {
      const int jc = pred_row4(p0 + p, (int)threadIdx.x, J);
      if (q_dtype == ETA_DT_F32) {
        const uint4 u = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint32_t*>(q) + qoff + jc);
        r.x[p][0] = u.x; r.x[p][1] = u.y; r.x[p][2] = u.z; r.x[p][3] = u.w;
      } else {
        const uint2 u = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(q) + qoff + jc);
        r.x[p][0] = u.x & 0xffffu; r.x[p][1] = u.x >> 16; r.x[p][2] = u.y & 0xffffu; r.x[p][3] = u.y >> 16;
      }
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int hc = h0 + (c < ncols ? c : 0);
        const float4 w4 = *reinterpret_cast<const float4*>(W + (int64_t)hc * J + jc);
        r.w[p][c][0] = w4.x; r.w[p][c][1] = w4.y; r.w[p][c][2] = w4.z; r.w[p][c][3] = w4.w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int jc = j + e < J ? j + e : 0;
        r.x[p][e] = q_dtype == ETA_DT_F32 ? reinterpret_cast<const uint32_t*>(q)[qoff + jc]
                                          : (uint32_t)reinterpret_cast<const uint16_t*>(q)[qoff + jc];
#pragma unroll
        for (int c = 0; c < NC; ++c) r.w[p][c][e] = W[(int64_t)(h0 + (c < ncols ? c : 0)) * J + jc];
      }
    }
  }
}

template <int NC>
__device__ __forceinline__ void pred_fma(int q_dtype, int J, int ncols, int p0,
                                         const PredRows<NC>& r, float (&acc)[NC]) {
#pragma unroll
  for (int p = 0; p < kPredPass; ++p) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool in = (p0 + p) * kPredStep + 4 * (int)threadIdx.x + e < J;
      const float x = in ? pred_x(r.x[p][e], q_dtype) : 0.f;
#pragma unroll
      for (int c = 0; c < NC; ++c) acc[c] = fmaf(x, (in && c < ncols) ? r.w[p][c][e] : 0.f, acc[c]);
    }
  }
}

// Thread t's partial sums over its rows in the order above: the first
// kPredPass passes from r (loaded by pred_load at pass 0), the rest loaded
// kPredPass passes at a time.
template <int NC, bool VEC>
__device__ __forceinline__ void pred_sum(const void* __restrict__ q, int q_dtype, int64_t qoff,
                                         const float* __restrict__ W, int J, int h0, int ncols,
                                         const PredRows<NC>& r, float (&acc)[NC]) {
#pragma unroll
  for (int c = 0; c < NC; ++c) acc[c] = 0.f;
  pred_fma<NC>(q_dtype, J, ncols, 0, r, acc);
  for (int p0 = kPredPass; p0 * kPredStep < J; p0 += kPredPass) {
    PredRows<NC> r2;
    pred_load<NC, VEC>(q, q_dtype, qoff, W, J, h0, ncols, p0, r2);
    pred_fma<NC>(q_dtype, J, ncols, p0, r2, acc);
  }
}

// Reduces the partials of the workgroup (kPredThreads threads); red holds
// [4][NC] floats.  Thread c < ncols gets column c's total in *tot (bias not added).
template <int NC>
__device__ __forceinline__ void pred_reduce(const float (&acc)[NC], int ncols, float* red,
                                            float* tot) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const float x = wave_sum(acc[c]);
    if (lane == 0) red[w * NC + c] = x;
  }
  __syncthreads();
  if ((int)threadIdx.x < ncols) {
    float t = 0.f;
#pragma unroll
    for (int k = 0; k < kPredThreads / 64; ++k) t += red[k * NC + threadIdx.x];
    *tot = t;
  }
  __syncthreads();
}

#if ETA_PART == 0
__global__ __launch_bounds__(kPredThreads) void predict_kernel(const void* __restrict__ q,
                                                               int q_dtype,
                                                               const float* __restrict__ W,
                                                               const float* __restrict__ bias,
                                                               float* __restrict__ tau, int Hq,
                                                               int D) {
  __shared__ float red[4 * kPredCols];
  const int b = blockIdx.x, h0 = blockIdx.y * kPredCols;
  const int ncols = Hq - h0 < kPredCols ? Hq - h0 : kPredCols;
  const int64_t J = (int64_t)Hq * D;
  float acc[kPredCols];
  if (W != nullptr && J % 4 == 0) {
    PredRows<kPredCols> rows;
    pred_load<kPredCols, true>(q, q_dtype, (int64_t)b * J, W, (int)J, h0, ncols, 0, rows);
    pred_sum<kPredCols, true>(q, q_dtype, (int64_t)b * J, W, (int)J, h0, ncols, rows, acc);
  } else if (W != nullptr) {
    PredRows<kPredCols> rows;
    pred_load<kPredCols, false>(q, q_dtype, (int64_t)b * J, W, (int)J, h0, ncols, 0, rows);
    pred_sum<kPredCols, false>(q, q_dtype, (int64_t)b * J, W, (int)J, h0, ncols, rows, acc);
  } else {
#pragma unroll
    for (int c = 0; c < kPredCols; ++c) acc[c] = 0.f;
  }
  float t = 0.f;
  pred_reduce<kPredCols>(acc, ncols, red, &t);
  if ((int)threadIdx.x < ncols) tau[(int64_t)b * Hq + h0 + threadIdx.x] = t + bias[h0 + threadIdx.x];
}
#endif

// ---------------------------------------------------------------- screening
//
// One workgroup of 256 threads per (tile of 64 blocks, kv head, sequence).
// Wavefront w takes head-dimension quarter w; with the dimension-major
// summaries, lane (cg, qd) (cg = lane / 16, qd = lane % 16) reads coordinate
// 4 k + cg of the tile's blocks 4 qd .. 4 qd + 3 with one load per record array,
// so a wavefront has 17 loads in flight for its quarter.  These loads are
// issued right after the threshold and query loads, and every later step waits
// only for its own.  The G query heads of the group are evaluated from the
// same loads (q broadcast from LDS).  The partial sums reach wavefront 0 (lane
// = block) through LDS; it adds them in a fixed order and owns everything per
// block after that: selection, the rescue part, mask, and the ordered
// compaction of the tile's union ids (one ballot).  A union id carries the
// block's head bits in its top byte.
//
// Top-1 rescue needs the selection state of the whole window [0, min(c, N)),
// which can span up to four tiles.  Each tile that meets the window writes its
// part: per head, whether one of its window blocks is selected, else the first
// of its largest bounds and that block; and the union head bits of its window
// blocks.  The split kernel, which runs after screening anyway, combines the
// parts, so no workgroup waits for another.
//
// With a predictor (W, bias), every workgroup computes the thresholds of its
// G heads itself, with the stand-alone predictor's summation order (so they
// are bit-identical to eta_predict_threshold's); tile 0 stores them.

struct ScreenArgs {
  const void* q;
  const int32_t* seq_lens;
  const float* tau;          // given thresholds, or nullptr with `predict`
  const float* W;            // predictor weights (may be nullptr: constants)
  const float* bias;
  float* tau_store;          // predicted thresholds for the decode kernel (tile 0 writes)
  float* tau_out;            // optional copy for the caller
  const void* mu;             // stat type ST
  const void* sigma;
  const float* mx;
  uint8_t* mask;
  int32_t* ids;
  int32_t* tile_cnt;
  int32_t* head_cnt;
  float* bounds;
  float* resc_best;          // [B][Hq][kRescueTiles] window part of each tile: largest bound
  int32_t* resc_info;        //   its block, kRescueNone, or kRescueAny (a window block selected)
  uint8_t* wbits;            // [B][Hkv][kMaxRescueWindow] union head bits of the window blocks
  Geom g;
  int q_dtype;
  int predict;
  float z, offset_a;
  int c, lwb, screen_all;
};

constexpr int kScreenThreads = 256;
constexpr uint32_t kIdMask = 0x00ffffffu;   // union id: block index | head bits << 24

// Tile of screening workgroup k.  With one-byte records a tile's coordinate row
// is 64 bytes, half a 128-byte line; workgroups are dealt to the eight XCDs
// (each with its own L2) round robin, so with the identity mapping the two
// halves of every line would be fetched by two XCDs.  When the grid's x extent
// is a multiple of 16 the mapping pairs tiles 2j and 2j + 1 on workgroups j and
// j + 8 of each group of 16, which land on the same XCD.
template <typename ST>
__device__ __forceinline__ int screen_tile(int k) {
  if constexpr (sizeof(ST) == 1) {
    if ((gridDim.x & 15u) == 0) return (k & ~15) | ((k & 7) << 1) | ((k >> 3) & 1);
  }
  return k;
}

template <int D, int G, bool BOUNDS_ONLY, typename ST, bool VEC>
__global__ __launch_bounds__(kScreenThreads) void screen_kernel(ScreenArgs a) {
  constexpr int DQ = D / 4;            // dimensions per quarter
  const Geom& g = a.g;
  const int tile = screen_tile<ST>(blockIdx.x), gh = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  __shared__ float q_s[D][G];
  __shared__ float q2_s[D][G];
  __shared__ float qn_s[G];
  __shared__ float teff_s[G];
  __shared__ float part_s[4][2 * G][kScreenTile];
  __shared__ float pred_red[4 * G];

  const int64_t hq0 = (int64_t)b * g.Hq + (int64_t)gh * G;   // first query head row of the group
  const int64_t bg = (int64_t)b * g.Hkv + gh;
  const float scale = 1.0f / sqrtf((float)D);
  const float z = a.z;

  // This lane's summary loads: coordinate w DQ + 4 k + cg (cg = lane / 16) of the
  // four consecutive blocks jb + 4 qd .. + 3 (qd = lane % 16), one load per
  // record array and k when the rows are four-record aligned (VEC: n_blk_cap a
  // multiple of 4), else four; indexes clamped into the buffers (records of
  // blocks that are not full are discarded later; n_blk_cap >= 1).  Wavefront 0
  // uses the largest norm of block jb + lane.
  constexpr int NK = DQ / 4;
  const int cg = lane >> 4, qd = lane & 15;
  auto issue = [&](int64_t jb, Rec4<ST> (&m)[NK], Rec4<ST> (&sd)[NK], float& M) {
    const int64_t row0 = bg * D + w * DQ + cg;
    if constexpr (VEC) {             // n_blk_cap >= 4, a multiple of 4
#pragma unroll
      for (int k = 0; k < NK; ++k) {
        const int64_t o = screen_rec4_offset(row0 + 4 * k, g.ncap, jb + 4 * qd);
        m[k] = *reinterpret_cast<const Rec4<ST>*>(reinterpret_cast<const ST*>(a.mu) + o);
        sd[k] = *reinterpret_cast<const Rec4<ST>*>(reinterpret_cast<const ST*>(a.sigma) + o);
      }
    } else {
#pragma unroll
      for (int k = 0; k < NK; ++k) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int64_t o = screen_rec1_offset(row0 + 4 * k, g.ncap, jb + 4 * qd + e);
          m[k].v[e] = reinterpret_cast<const ST*>(a.mu)[o];
          sd[k].v[e] = reinterpret_cast<const ST*>(a.sigma)[o];
        }
      }
    }
    int64_t jm = jb + lane;
    jm = jm < g.ncap ? jm : g.ncap - 1;
    M = a.mx[bg * g.ncap + jm];       // (used by wavefront 0)
  };
  // the bias (or given threshold) and the predictor rows first, then this
  // tile's summaries: each is consumed in that order, so no wait for a later
  // load holds up an earlier step
  const int64_t T = clamp_len(a.seq_lens, b, g.cap);
  float tau_in = 0.f;
  if (!BOUNDS_ONLY && tid < G) tau_in = a.predict ? a.bias[gh * G + tid] : a.tau[hq0 + tid];
  // this wavefront's query elements: heads w, w + 4, ..., dimensions lane + 64 s
  constexpr int QH = (G + 3) / 4, QI = D / 64;
  uint32_t qraw[QH][QI];
#pragma unroll
  for (int r = 0; r < QH; ++r) {
    const int h = w + 4 * r < G ? w + 4 * r : 0;
#pragma unroll
    for (int si = 0; si < QI; ++si) {
      const int64_t idx = (hq0 + h) * D + lane + 64 * si;
      qraw[r][si] = a.q_dtype == ETA_DT_F32 ? reinterpret_cast<const uint32_t*>(a.q)[idx]
                                            : (uint32_t)reinterpret_cast<const uint16_t*>(a.q)[idx];
    }
  }
  const bool predict = !BOUNDS_ONLY && a.predict && a.W != nullptr;
  const int64_t Jq = (int64_t)g.Hq * D;
  PredRows<G> prow;
  // the group's G rows of W (Hq d is a multiple of 4 here: d is 64 or 128)
  if (predict) pred_load<G, true>(a.q, a.q_dtype, (int64_t)b * Jq, a.W, (int)Jq, gh * G, G, 0, prow);
  Rec4<ST> m0[NK], sd0[NK];
  float M0;
  issue((int64_t)tile * kScreenTile, m0, sd0, M0);

  // the group's queries, their norms (one wavefront per head), thresholds
#pragma unroll
  for (int r = 0; r < QH; ++r) {
    const int h = w + 4 * r;
    if (h < G) {
      float ss = 0.f;
#pragma unroll
      for (int si = 0; si < QI; ++si) {
        const int i = lane + 64 * si;
        const float x = pred_x(qraw[r][si], a.q_dtype);
        q_s[i][h] = x;
        q2_s[i][h] = x * x;
        ss = fmaf(x, x, ss);
      }
      ss = wave_sum(ss);
      if (lane == 0) qn_s[h] = sqrtf(ss);
    }
  }
  // predictor: this wavefront's partial sums of the group's G columns (the
  // wavefronts' partials are added after the barrier below, in the stand-alone
  // predictor's order, so the thresholds are bit-identical to it)
  if constexpr (!BOUNDS_ONLY) {
    if (predict) {
      float acc[G];
      pred_sum<G, true>(a.q, a.q_dtype, (int64_t)b * Jq, a.W, (int)Jq, gh * G, G, prow, acc);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float x = wave_sum(acc[h]);
        if (lane == 0) pred_red[w * G + h] = x;
      }
    }
  }
  __syncthreads();
  // thresholds: read by the selection only, after the barriers in `finish`
  if constexpr (!BOUNDS_ONLY) {
    if (tid < G) {
      float tau = tau_in;
      if (a.predict) {
        float t = 0.f;
        if (predict) {
#pragma unroll
          for (int k = 0; k < 4; ++k) t += pred_red[k * G + tid];
        }
        tau = t + tau_in;
        if (tile == 0) {
          a.tau_store[hq0 + tid] = tau;
          if (a.tau_out != nullptr) a.tau_out[hq0 + tid] = tau;
        }
      } else if (tile == 0 && a.tau_out != nullptr) {
        a.tau_out[hq0 + tid] = tau;   // thresholds predicted by predict_kernel
      }
      teff_s[tid] = tau - a.offset_a;
    }
  }

  const int64_t N = T / g.BS;

  // Bounds of blocks jb + lane from loads issued by `issue` (all four
  // wavefronts take part); valid in wavefront 0, NaN for blocks not full.  Each
  // lane sums its coordinates in order; the four coordinate groups of a block
  // are added by row swaps (two registers per swap: block 4 qd + r of the quad
  // ends in row r, as partial sums (rows 0 + 1) + (rows 2 + 3)); wavefront 0
  // adds the four wavefronts' partials in order.
  auto finish = [&](int64_t jb, const Rec4<ST> (&m)[NK], const Rec4<ST> (&sd)[NK], float M,
                    float (&bnd)[G]) {
    const int64_t j = jb + lane;
    float dot[G][4], var[G][4];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 4; ++e) { dot[h][e] = 0.f; var[h][e] = 0.f; }
#pragma unroll
    for (int k = 0; k < NK; ++k) {
      // keep the query's LDS reads inside the loop (hoisted they hold registers)
      asm volatile("" ::: "memory");
      const int i = w * DQ + 4 * k + cg;
      float mv[4], sv[4];
      rec4_f32(m[k], mv);
      rec4_f32(sd[k], sv);
#pragma unroll
      for (int e = 0; e < 4; ++e) sv[e] *= sv[e];
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float qh = q_s[i][h], q2 = q2_s[i][h];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          dot[h][e] = fmaf(qh, mv[e], dot[h][e]);
          var[h][e] = fmaf(q2, sv[e], var[h][e]);
        }
      }
    }
    auto sum16 = [](float x, float y) {
      const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(y), false, false);
      return __uint_as_float(r[0]) + __uint_as_float(r[1]);
    };
    auto sum32 = [](float x, float y) {
      const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(y), false, false);
      return __uint_as_float(r[0]) + __uint_as_float(r[1]);
    };
    const int jq = 4 * qd + cg;       // the block whose sums this lane ends with
#pragma unroll
    for (int h = 0; h < G; ++h) {
      part_s[w][h][jq] = sum32(sum16(dot[h][0], dot[h][1]), sum16(dot[h][2], dot[h][3]));
      part_s[w][G + h][jq] = sum32(sum16(var[h][0], var[h][1]), sum16(var[h][2], var[h][3]));
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < G; ++h) bnd[h] = __builtin_nanf("");
    if (w == 0 && j < N) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float dt = ((part_s[0][h][lane] + part_s[1][h][lane]) + part_s[2][h][lane]) +
                         part_s[3][h][lane];
        const float vr = ((part_s[0][G + h][lane] + part_s[1][G + h][lane]) +
                          part_s[2][G + h][lane]) + part_s[3][G + h][lane];
        const float gauss = fmaf(z, sqrtf(vr), dt);
        const float spher = qn_s[h] * M;
        float lo = gauss < spher ? gauss : spher;
        if (isnan(gauss) || isnan(spher)) lo = __builtin_nanf("");
        bnd[h] = lo * scale;
      }
    }
    __syncthreads();
  };

  const int64_t j = (int64_t)tile * kScreenTile + lane;
  float bnd[G];
  finish((int64_t)tile * kScreenTile, m0, sd0, M0, bnd);

  if constexpr (BOUNDS_ONLY) {
    if (w == 0 && j < g.ncap) {
#pragma unroll
      for (int h = 0; h < G; ++h) a.bounds[(hq0 + h) * g.ncap + j] = bnd[h];
    }
    return;
  } else {
    auto selected = [&](int64_t jj, float bd, int h) {
      return jj < N && (a.screen_all || bd >= teff_s[h] || jj >= N - a.lwb);
    };
    uint32_t bits = 0;
#pragma unroll
    for (int h = 0; h < G; ++h) bits |= (uint32_t)selected(j, bnd[h], h) << h;

    if (w != 0) return;
    // top-1 rescue over the window [0, min(c, N)): this tile's part of it, per
    // head whether any of its window blocks is selected and the first of its
    // largest non-NaN bounds, and the union head bits of its window blocks; the
    // split kernel combines the window's tiles and attends the rescued block
    const int64_t Wn = (int64_t)a.c < N ? (int64_t)a.c : N;
    if (a.c > 0 && (int64_t)tile * kScreenTile < Wn) {
      const bool inw = j < Wn;
      float bv[G];
      int bi[G];
      bool any[G];
#pragma unroll
      for (int h = 0; h < G; ++h) {
        any[h] = __ballot(inw && ((bits >> h) & 1u)) != 0ull;
        const bool ok = inw && !isnan(bnd[h]);
        bv[h] = ok ? bnd[h] : kNegInf;
        bi[h] = ok ? (int)j : 0x7fffffff;
      }
      wave_argmax_n<G>(bv, bi);
      if (lane == 0) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const int64_t e = (hq0 + h) * kRescueTiles + tile;
          a.resc_best[e] = bv[h];
          a.resc_info[e] = any[h] ? kRescueAny : (bi[h] == 0x7fffffff ? kRescueNone : bi[h]);
        }
      }
      if (inw) a.wbits[bg * kMaxRescueWindow + j] = (uint8_t)bits;
    }
    if (j < g.ncap) {
#pragma unroll
      for (int h = 0; h < G; ++h) a.mask[(hq0 + h) * g.ncap + j] = (uint8_t)((bits >> h) & 1u);
    }
    // ordered compaction of the tile's union ids and the per-head counts
    const unsigned long long bal = __ballot(bits != 0);
    if (bits != 0) a.ids[union_slot(bg * g.ncap, tile, bal, lane)] = (int32_t)((uint32_t)j | (bits << 24));
    if (lane == 0) a.tile_cnt[bg * g.n_tiles + tile] = __popcll(bal);
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const unsigned long long bh = __ballot((bits >> h) & 1u);
      if (lane == 0) a.head_cnt[(hq0 + h) * g.n_tiles + tile] = __popcll(bh);
    }
  }
}

// ---------------------------------------------------------------- split decode
//
// One workgroup (kSplitWaves wavefronts) per (split, kv head, sequence).  Split
// s of S owns the (sequence, kv head)'s union-list tiles of 64 tokens s, s + S,
// s + 2 S, ... (bf16; a contiguous range of whole blocks for fp32), so shares
// differ by at most one tile; wavefront w takes its share's tiles w,
// w + kSplitWaves, ...  A block is processed 64 tokens at a time,
// lane = token for the scores (each lane reads its own K row with 16-byte
// loads) and lane = head-dimension pair for p.V (coalesced rows of V), with
// the weights p passed through the wavefront's LDS slice.  A head skips blocks
// it did not select even when a sibling head of the group loaded them (the
// union is loaded once, each head keeps its own online-softmax state).  The
// last split also attends the partial tail.  The four wavefront states are
// merged through LDS into one partial (max, sum, acc) per head and split.

// bf16 V rows in the split kernels: each wavefront load reads whole rows (128
// or 256 bytes), each read once per step, so they are loaded with the
// non-temporal hint and do not displace the lines that the K loads (16-byte
// pieces of 64 rows per load, merged into whole lines by the caches) and the
// next step's index reads still use: at 512K / 20% this took split decode from
// 111 to 99 us.  K keeps the default policy (with the hint the same kernel took
// 198 us).
__device__ __forceinline__ uint32_t load_v_pair(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p));
}
__device__ __forceinline__ uint16_t load_v_one(const uint16_t* p) {
  return __builtin_nontemporal_load(p);
}

// Scores of bf16 K on the matrix cores: v_mfma_f32_16x16x32_bf16 with a
// block-diagonal A.  Row m = 4*tg + h of A holds query head h restricted to the
// k-slots of lane group tg, so the 16x16 result hands lane l the G <= 4 head
// scores of token l; the B operand is exactly each lane's own K row chunk.
// G = 8 runs two head quads.  fp32 q is split into bf16 hi + lo parts (two
// MFMAs) so the scores keep ~16 mantissa bits; fp32 K uses the vector ALUs.


}  // namespace

struct SplitArgs {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* seq_lens;
  const float* tau;
  const int32_t* ids;
  const int32_t* tile_cnt;
  float2* part_ml;           // [splits][G] (max, sum) per split workgroup and head
  float* part_acc;           // [splits][G][D]
  const float* resc_best;    // screening's window parts (see ScreenArgs)
  const int32_t* resc_info;
  const uint8_t* wbits;
  uint8_t* mask;             // the rescued blocks' mask bits are set here
  int32_t* resc_out;         // [B][Hq] rescued block per head, or -1 (for the combine)
  int32_t* extra_union;      // [B][Hkv] rescued blocks outside the union (for the combine)
  int2* plan;                // [B][Hkv] (first split workgroup, splits) of each group
  // one split per group (uniform plan, S = 1): the split writes the final
  // results itself and no combine runs
  const int32_t* head_cnt;   // [B][Hq][n_tiles] selected blocks per head per tile
  void* out;                 // [B][Hq][D] in q's type
  int32_t* counts;           // [B][Hq] attended tokens (may be nullptr)
  int32_t* union_counts;     // [B][Hkv] union blocks (may be nullptr)
  Geom g;
  int q_dtype;
  float beta, offset_a;
  int self_ungated;
  int c;                     // rescue window (blocks)
};

namespace {


// Gated score S~ = S sigmoid(beta (S - tau_eff)); -inf when the head does not
// attend the token.
template <bool DENSE>
__device__ __forceinline__ float gated(float S, bool attend, bool ungated, float teff, float beta) {
  if (!attend) return kNegInf;
  if (DENSE || ungated || teff == kNegInf) return S;
  return S * __builtin_amdgcn_rcpf(1.0f + __expf(-beta * (S - teff)));
}

// Online-softmax update of one head with this lane's score `sc`; returns the
// lane's weight and rescales the head's accumulator.
template <int DPL>
__device__ __forceinline__ float softmax_step(float sc, float& m, float& l, float (&acc)[DPL]) {
  const float bm = wave_max(sc);
  const float mn = fmaxf(m, bm);
  if (mn == kNegInf) return 0.f;
  const float alpha = __expf(m - mn);
  const float p = __expf(sc - mn);
  l = l * alpha + wave_sum(p);
  m = mn;
#pragma unroll
  for (int e = 0; e < DPL; ++e) acc[e] *= alpha;
  return p;
}

// fp32 K/V: scores on the vector ALUs.
template <int D, int G, bool DENSE>
__device__ __forceinline__ void attend_f32(const float* __restrict__ kb, const float* __restrict__ vb,
                                           int64_t st, int64_t t0, int nvalid, uint32_t bits,
                                           const float (*qf_s)[G], const float* teff_s,
                                           float (*p_s)[G], float beta, int64_t self_t, int lane,
                                           float (&m_)[G], float (&l_)[G], float (&acc)[G][D / 64]) {
  constexpr int DPL = D / 64;
  for (int sb = 0; sb < nvalid; sb += 64) {
    asm volatile("" ::: "memory");
    const int nv = nvalid - sb < 64 ? nvalid - sb : 64;
    const bool valid = lane < nv;
    const int64_t row = t0 + sb + (valid ? lane : 0);
    float dot[G];
#pragma unroll
    for (int h = 0; h < G; ++h) dot[h] = 0.f;
#pragma unroll 2
    for (int i = 0; i < D; i += 8) {
      float x[8];
      Elem<float>::load8(kb + row * st + i, x);
#pragma unroll
      for (int e = 0; e < 8; ++e)
#pragma unroll
        for (int h = 0; h < G; ++h) dot[h] = fmaf(x[e], qf_s[i + e][h], dot[h]);
    }
    const bool ung = (t0 + sb + lane) == self_t;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float sc = gated<DENSE>(dot[h], valid && ((bits >> h) & 1u), ung, teff_s[h], beta);
      p_s[lane][h] = softmax_step<DPL>(sc, m_[h], l_[h], acc[h]);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    for (int t = 0; t < nv; ++t) {
      float vv[DPL];
      Elem<float>::template loadn<DPL>(vb + (t0 + sb + t) * st + lane * DPL, vv);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float ph = p_s[t][h];
#pragma unroll
        for (int e = 0; e < DPL; ++e) acc[h][e] = fmaf(ph, vv[e], acc[h][e]);
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// bf16 K/V: scores on the matrix cores.
template <int D, int G, bool DENSE>
__device__ __forceinline__ void attend_bf16(const uint16_t* __restrict__ kb,
                                            const uint16_t* __restrict__ vb, int64_t st, int64_t t0,
                                            int nvalid, uint32_t bits, const bf16x8* qa_s,
                                            bool use_lo, const float* teff_s, float* p_s,
                                            float beta, float scale, int64_t self_t, int lane,
                                            float (&m_)[G], float (&l_)[G],
                                            float (&acc)[G][D / 64]) {
  constexpr int DPL = D / 64;
  constexpr int DC = D / 8;               // 16-byte chunks per row = MFMAs per head quad
  constexpr int NQ = G > 4 ? G / 4 : 1;   // head quads
  constexpr int GQ = 4 * NQ;              // padded heads (LDS row of p)
  const bool diag = ((lane & 15) >> 2) == (lane >> 4);
  const int qrow = lane & 3;
  for (int sb = 0; sb < nvalid; sb += 64) {
    asm volatile("" ::: "memory");
    const int nv = nvalid - sb < 64 ? nvalid - sb : 64;
    const bool valid = lane < nv;
    const int64_t tb = t0 + sb;
    // issue every load of the 64-token step first: this lane's K row and, for
    // every token, this lane's head-dimension pair of V (rows past the valid
    // ones read token tb again and get weight 0)
    uint4 kr[DC];
    const uint16_t* krow = kb + (tb + (valid ? lane : 0)) * st;
#pragma unroll
    for (int c = 0; c < DC; ++c) kr[c] = *reinterpret_cast<const uint4*>(krow + 8 * c);
    uint32_t vr[64];
#pragma unroll
    for (int t = 0; t < 64; ++t) {
      const int64_t r = tb + (t < nv ? t : 0);
      if constexpr (DPL == 2)
        vr[t] = load_v_pair(vb + r * st + 2 * lane);
      else
        vr[t] = load_v_one(vb + r * st + lane);
    }
    const bool ung = (tb + lane) == self_t;
#pragma unroll
    for (int hq = 0; hq < NQ; ++hq) {
      f32x4 c = {0.f, 0.f, 0.f, 0.f};
      const bf16x8 zero = {};
#pragma unroll
      for (int ch = 0; ch < DC; ++ch) {
        const bf16x8 bk = __builtin_bit_cast(bf16x8, kr[ch]);
        const bf16x8 ahi = diag ? qa_s[((hq * 2 + 0) * 4 + qrow) * DC + ch] : zero;
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, bk, c, 0, 0, 0);
        if (use_lo) {
          const bf16x8 alo = diag ? qa_s[((hq * 2 + 1) * 4 + qrow) * DC + ch] : zero;
          c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, bk, c, 0, 0, 0);
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int h = 4 * hq + r;
        if (h < G) {
          const float sc =
              gated<DENSE>(c[r] * scale, valid && ((bits >> h) & 1u), ung, teff_s[h], beta);
          p_s[lane * GQ + h] = softmax_step<DPL>(sc, m_[h], l_[h], acc[h]);
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int t = 0; t < 64; ++t) {
      float vv[DPL];
      if constexpr (DPL == 2) {
        vv[0] = bf16lo(vr[t]);
        vv[1] = bf16hi(vr[t]);
      } else {
        vv[0] = bf16lo(vr[t]);
      }
#pragma unroll
      for (int hq = 0; hq < NQ; ++hq) {
        const float4 p4 = *reinterpret_cast<const float4*>(p_s + t * GQ + 4 * hq);
        const float pr[4] = {p4.x, p4.y, p4.z, p4.w};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int h = 4 * hq + r;
          if (h < G) {
#pragma unroll
            for (int e = 0; e < DPL; ++e) acc[h][e] = fmaf(pr[r], vv[e], acc[h][e]);
          }
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// bf16 K/V, full 64-token tiles of one wavefront, software-pipelined: the next
// tile's K loads are issued as soon as this tile's MFMAs have consumed the K
// registers, and its V loads as soon as p.V has consumed the V registers, so
// each wavefront keeps about one tile of K and V in flight while it computes.
// tile_base(u) gives the first token of tile u, tile_bits(u) its head mask.
template <int D, int G, bool DENSE, typename TB, typename BITS>
__device__ __forceinline__ void attend_bf16_stream(const uint16_t* __restrict__ kb,
                                                   const uint16_t* __restrict__ vb, int64_t st,
                                                   int ntiles, TB tile_base, BITS tile_bits,
                                                   const bf16x8* qa_s, bool use_lo,
                                                   const float* teff_s, float* p_s, float beta,
                                                   float scale, int64_t self_t, int lane,
                                                   float (&m_)[G], float (&l_)[G],
                                                   float (&acc)[G][D / 64]) {
  constexpr int DPL = D / 64;
  constexpr int DC = D / 8;
  constexpr int NQ = G > 4 ? G / 4 : 1;
  constexpr int GQ = 4 * NQ;
  if (ntiles <= 0) return;
  const bool diag = ((lane & 15) >> 2) == (lane >> 4);
  const int qrow = lane & 3;
  uint4 kr[DC];
  uint32_t vr[64];
  auto load_k = [&](int64_t tb) {
    const uint16_t* krow = kb + (tb + lane) * st;
#pragma unroll
    for (int c = 0; c < DC; ++c) kr[c] = *reinterpret_cast<const uint4*>(krow + 8 * c);
  };
  auto load_v_rows = [&](int64_t tb, int t0) {
#pragma unroll
    for (int t = t0; t < t0 + 16; ++t) {
      if constexpr (DPL == 2)
        vr[t] = load_v_pair(vb + (tb + t) * st + 2 * lane);
      else
        vr[t] = load_v_one(vb + (tb + t) * st + lane);
    }
  };
  auto load_v = [&](int64_t tb) {
#pragma unroll
    for (int qt = 0; qt < 4; ++qt) load_v_rows(tb, 16 * qt);
  };
  // One tile: scores on the MFMAs, then (MORE) the next tile's K loads into the
  // freed K registers, the softmax update, p.V, then (MORE) the next tile's V
  // loads.  The last tile is peeled (MORE = false) so that the loads inside the
  // loop are unconditional: a conditional reload would keep two copies of the
  // K/V registers alive across the branch.
  auto tile = [&](int u, int64_t tb, int64_t tbn, auto more_tag) {
    constexpr bool MORE = decltype(more_tag)::value;
    asm volatile("" ::: "memory");
    const uint32_t bits = tile_bits(u);
    const bool ung = (tb + lane) == self_t;
    f32x4 c[NQ];
#pragma unroll
    for (int hq = 0; hq < NQ; ++hq) {
      c[hq] = f32x4{0.f, 0.f, 0.f, 0.f};
      const bf16x8 zero = {};
#pragma unroll
      for (int ch = 0; ch < DC; ++ch) {
        const bf16x8 bk = __builtin_bit_cast(bf16x8, kr[ch]);
        const bf16x8 ahi = diag ? qa_s[((hq * 2 + 0) * 4 + qrow) * DC + ch] : zero;
        c[hq] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, bk, c[hq], 0, 0, 0);
        if (use_lo) {
          const bf16x8 alo = diag ? qa_s[((hq * 2 + 1) * 4 + qrow) * DC + ch] : zero;
          c[hq] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, bk, c[hq], 0, 0, 0);
        }
      }
    }
    if constexpr (MORE) {
      __builtin_amdgcn_sched_barrier(0);
      load_k(tbn);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int hq = 0; hq < NQ; ++hq) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int h = 4 * hq + r;
        if (h < G) {
          const float sc = gated<DENSE>(c[hq][r] * scale, (bits >> h) & 1u, ung, teff_s[h], beta);
          p_s[lane * GQ + h] = softmax_step<DPL>(sc, m_[h], l_[h], acc[h]);
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    // p.V in four quarters of 16 tokens; as soon as a quarter's V registers
    // are consumed, that quarter of the next tile's V rows is requested, so
    // those loads overlap the rest of this tile and the next tile's scores
#pragma unroll
    for (int qt = 0; qt < 4; ++qt) {
#pragma unroll
      for (int t = 16 * qt; t < 16 * qt + 16; ++t) {
        float vv[DPL];
        if constexpr (DPL == 2) {
          vv[0] = bf16lo(vr[t]);
          vv[1] = bf16hi(vr[t]);
        } else {
          vv[0] = bf16lo(vr[t]);
        }
#pragma unroll
        for (int hq = 0; hq < NQ; ++hq) {
          const float4 p4 = *reinterpret_cast<const float4*>(p_s + t * GQ + 4 * hq);
          const float pr[4] = {p4.x, p4.y, p4.z, p4.w};
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int h = 4 * hq + r;
            if (h < G) {
#pragma unroll
              for (int e = 0; e < DPL; ++e) acc[h][e] = fmaf(pr[r], vv[e], acc[h][e]);
            }
          }
        }
      }
      if constexpr (MORE) {
        __builtin_amdgcn_sched_barrier(0);
        load_v_rows(tbn, 16 * qt);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    __builtin_amdgcn_wave_barrier();
  };
  int64_t tb = tile_base(0);
  load_k(tb);
  load_v(tb);
  for (int u = 0; u + 1 < ntiles; ++u) {
    const int64_t tbn = tile_base(u + 1);
    tile(u, tb, tbn, std::integral_constant<bool, true>{});
    tb = tbn;
  }
  tile(ntiles - 1, tb, tb, std::integral_constant<bool, false>{});
}

constexpr int kItemChunk = 256;
// Wavefronts per split-decode workgroup.
constexpr int kSplitWaves = 4;

template <int D, int BS, int G, typename KVT, bool DENSE, bool PROP>
__global__ __launch_bounds__(64 * kSplitWaves) void split_kernel(SplitArgs a) {
  constexpr int NW = kSplitWaves, NT = 64 * NW;
  constexpr int DPL = D / 64;
  constexpr bool BF = sizeof(KVT) == 2;
  constexpr int NQ = G > 4 ? G / 4 : 1;
  constexpr int GQ = 4 * NQ;
  constexpr int DC = D / 8;
  const Geom& g = a.g;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  __shared__ float qf_s[BF ? 1 : D][G];                  // fp32 path: scaled q
  __shared__ bf16x8 qa_s[BF ? NQ * 2 * 4 * DC : 1];      // bf16 path: q chunks (hi, lo)
  __shared__ float teff_s[G];
  __shared__ int pref_s[kMaxTiles + 1];
  __shared__ int wsum_s[NW];
  __shared__ float mrg_ml[NW][G][2];
  __shared__ float mrg_acc[NW][G][D];
  __shared__ __attribute__((aligned(16))) float p_s[NW][64 * GQ];
  __shared__ int32_t item_j[kItemChunk];
  __shared__ uint8_t item_bits[kItemChunk];
  __shared__ uint8_t item_sub[kItemChunk];
  __shared__ int own_s[3];                               // proportional: (group, first split, splits)
  __shared__ int wsum2_s[DENSE ? 1 : kPropMaxGroups / NT][NW];  // proportional: split scan's wavefront sums
  __shared__ int cnt_s[DENSE ? 1 : kPropMaxCounts + 1];  // proportional: prefix of every tile count
  __shared__ int wtail_s[NW];
  __shared__ float rbest_s[DENSE ? 1 : G][kRescueTiles];
  __shared__ int rinfo_s[DENSE ? 1 : G][kRescueTiles];
  __shared__ int resc_s[G];                              // rescued block per head, or -1
  __shared__ int rx_s[G][2];                             // distinct rescued blocks: (block, heads)
  __shared__ int rxw_s[G];                               // union bits at each head's rescued block
  __shared__ int nrx_s;

  // ---- which (sequence, kv head) and split.  Uniform plan (PROP false): S splits
  // per group, grid (S, Hkv, B).  Proportional plan (PROP, several sequences): a
  // 1-D grid whose workgroups are dealt to the groups in proportion to their
  // union's 64-token tiles (at least one each), so short and long unions finish
  // together in one round.  The two plans are separate instantiations, so neither
  // carries the other's code.
  constexpr int SPB = BF ? BS / 64 : 1;
  constexpr bool uniform = !PROP;
  static_assert(!(DENSE && PROP), "the dense baseline takes the uniform plan");
  int b, gh, s, S, first;
  const int32_t* tc = nullptr;     // uniform: the group's tile counts
  const int* pref = pref_s;        // exclusive prefix of the group's tile counts ...
  int pbase = 0;                   // ... offset by pbase
  if constexpr (uniform) {
    s = blockIdx.x;
    gh = blockIdx.y;
    b = blockIdx.z;
    S = gridDim.x;
    first = (b * g.Hkv + gh) * S;
    tc = a.tile_cnt + ((int64_t)b * g.Hkv + gh) * g.n_tiles;
  } else {
    // Every tile count and every length in one round trip.  One block scan of
    // the counts (groups in order, each group's tiles in order) gives each
    // group's union tiles and, offset by the group's start, its own tile prefix;
    // a second scan over the groups' split counts gives each group's first split.
    const int BG = g.B * g.Hkv, nct = g.n_tiles, nc = BG * nct, W = gridDim.x;
    constexpr int CPT = kPropMaxCounts / NT;   // counts per thread, contiguous
    constexpr int GPT = kPropMaxGroups / NT;   // groups per thread: r NT + tid, r < GPT
    static_assert(CPT * NT == kPropMaxCounts && GPT * NT == kPropMaxGroups, "whole shares");
    // (unconditional loads from clamped indexes, masked afterwards: a load under a
    // branch is waited for inside the branch, one round trip each)
    int cv[CPT], tails[GPT];
#pragma unroll
    for (int k = 0; k < CPT; ++k) {
      const int i = tid * CPT + k;
      cv[k] = a.tile_cnt[i < nc ? i : 0];
    }
    {
      // group x = r NT + tid is (sequence x / Hkv, kv head x % Hkv)
      GroupStepper gs((unsigned)tid, (unsigned)NT, (unsigned)g.Hkv);
#pragma unroll
      for (int r = 0; r < GPT; ++r) {
        tails[r] = a.seq_lens[r * NT + tid < BG ? gs.q : 0u];
        gs.next();
      }
    }
    // every value is needed here, so none of the loads is moved into a branch
#pragma unroll
    for (int r = 0; r < GPT; ++r) asm volatile("" ::"v"(tails[r]));
#pragma unroll
    for (int k = 0; k < CPT; ++k)
      if (tid * CPT + k >= nc) cv[k] = 0;
    int ntl = 0;
#pragma unroll
    for (int r = 0; r < GPT; ++r) {
      const int x = r * NT + tid;
      const int64_t len = tails[r] < 0 ? 0 : (tails[r] > g.cap ? g.cap : tails[r]);
      // a group's work is its union's tiles plus one for a partial tail
      tails[r] = x < BG ? group_work(0, SPB, len, BS) : 0;
      ntl += tails[r];
    }
    int run = 0;
#pragma unroll
    for (int k = 0; k < CPT; ++k) {
      const int v = cv[k];
      cv[k] = run;
      run += v;
    }
    const int incl = wave_incl_scan(run);
    ntl = __builtin_amdgcn_readlane(wave_incl_scan(ntl), 63);
    if (lane == 63) wsum_s[w] = incl;
    if (lane == 0) wtail_s[w] = ntl;
    if (tid == 0) own_s[0] = -1;            // no group yet (set after two more barriers)
    __syncthreads();
    int woff = 0, tot = 0, ntails = 0;
#pragma unroll
    for (int k = 0; k < NW; ++k) {
      woff += k < w ? wsum_s[k] : 0;
      tot += wsum_s[k];
      ntails += wtail_s[k];
    }
    const int ex = woff + incl - run;
#pragma unroll
    for (int k = 0; k < CPT; ++k) cnt_s[tid * CPT + k] = ex + cv[k];
    if (tid == NT - 1) cnt_s[kPropMaxCounts] = ex + run;
    __syncthreads();
    // splits per group (integer work: the total does not depend on the order)
    const int64_t UT = (int64_t)tot * SPB + ntails;
    int nsp[GPT], inc[GPT];
#pragma unroll
    for (int r = 0; r < GPT; ++r) {
      const int x = r * NT + tid;
      nsp[r] = x < BG ? group_splits((cnt_s[(x + 1) * nct] - cnt_s[x * nct]) * SPB + tails[r],
                                     UT, W, BG)
                      : 0;
    }
    // one scan per round of NT groups in use
#pragma unroll
    for (int r = 0; r < GPT; ++r) inc[r] = r * NT < BG ? wave_incl_scan(nsp[r]) : 0;
    if (lane == 63) {
#pragma unroll
      for (int r = 0; r < GPT; ++r) wsum2_s[r][w] = inc[r];
    }
    __syncthreads();
    // group r NT + tid starts after every group of the earlier rounds, of the
    // earlier wavefronts of its round and of the earlier lanes; the workgroup's
    // group is the one whose splits include it (at most one thread finds it,
    // none for workgroups past the allocation)
    const int me = (int)blockIdx.x;
    int carry = 0;
#pragma unroll
    for (int r = 0; r < GPT; ++r) {
      int woff2 = 0, rt = 0;
#pragma unroll
      for (int k = 0; k < NW; ++k) {
        woff2 += k < w ? wsum2_s[r][k] : 0;
        rt += wsum2_s[r][k];
      }
      const int x = r * NT + tid, f = carry + woff2 + inc[r] - nsp[r];
      if (x < BG && owns_split(f, nsp[r], me)) {
        own_s[0] = x;
        own_s[1] = f;
        own_s[2] = nsp[r];
      }
      carry += rt;
    }
    __syncthreads();
    const int bgi = own_s[0];
    if (bgi < 0) return;             // workgroups past the allocation (uniform exit)
    b = bgi / g.Hkv;
    gh = bgi % g.Hkv;
    first = own_s[1];
    s = me - first;
    S = own_s[2];
    pref = cnt_s + bgi * nct;
    pbase = pref[0];
  }
  const int64_t hq0 = (int64_t)b * g.Hq + (int64_t)gh * G;
  const int64_t bg = (int64_t)b * g.Hkv + gh;
  const bool single = uniform && S == 1;             // no partials, no combine
  const float scale = 1.0f / sqrtf((float)D);
  // The independent loads go out together: length, the first 256 tile counts,
  // thresholds, the rescue window's parts and the query elements (as raw bits,
  // converted afterwards, so that no conversion waits on its own load).  The
  // rescue parts of every window tile are read (those past the window are never
  // used), so that no load waits for the length.
  int32_t t_raw = a.seq_lens[b];
  const int tc0 = (!DENSE && uniform && tid < g.n_tiles) ? tc[tid] : 0;
  const float tau_in = (!DENSE && tid < G) ? a.tau[hq0 + tid] : 0.f;
  float rb_in = 0.f;
  int ri_in = 0;
  if constexpr (!DENSE) {
    const int e = tid < G * kRescueTiles ? tid : 0;
    rb_in = a.resc_best[hq0 * kRescueTiles + e];
    ri_in = a.resc_info[hq0 * kRescueTiles + e];
  }
  constexpr int QE = BF ? NQ * 4 * D : G * D;          // staged query elements
  constexpr int QR = (QE + NT - 1) / NT;
  uint32_t qraw[QR];
#pragma unroll
  for (int r = 0; r < QR; ++r) {
    const int idx = tid + NT * r;
    const int hh = idx / D, i = idx % D;
    const int64_t src = (hq0 + ((idx < QE && hh < G) ? hh : 0)) * D + i;
    qraw[r] = a.q_dtype == ETA_DT_F32 ? reinterpret_cast<const uint32_t*>(a.q)[src]
                                      : (uint32_t)reinterpret_cast<const uint16_t*>(a.q)[src];
  }
  // the length and the rescue parts are taken here, after every load has been
  // issued (a uniform load is otherwise moved to a scalar register, with its
  // wait, right where it is issued)
  asm volatile("" : "+v"(t_raw) : "v"(rb_in), "v"(ri_in));
  t_raw = __builtin_amdgcn_readfirstlane(t_raw);
  const int64_t T = t_raw < 0 ? 0 : (t_raw > g.cap ? g.cap : (int64_t)t_raw);
  const int64_t N = T / BS;
  const int64_t Wn = (int64_t)a.c < N ? (int64_t)a.c : N;
  const int nwt = (int)((Wn + kScreenTile - 1) / kScreenTile);    // window tiles
  if constexpr (!DENSE) {
    if (tid < G * kRescueTiles) {
      rbest_s[tid / kRescueTiles][tid % kRescueTiles] = rb_in;
      rinfo_s[tid / kRescueTiles][tid % kRescueTiles] = ri_in;
    }
  }
  const int ntail = (int)(T - N * BS);
#pragma unroll
  for (int r = 0; r < QR; ++r) {
    const int idx = tid + NT * r;
    if (idx < QE) {
      const int hh = idx / D, i = idx % D;
      const float x = hh < G ? (a.q_dtype == ETA_DT_F32 ? __uint_as_float(qraw[r])
                                                        : __uint_as_float(qraw[r] << 16))
                             : 0.f;
      if constexpr (BF) {
        // chunk (quad, part, head r, c) = 8 bf16 of query head 4 quad + r, dims 8c..8c+7
        uint16_t* qa16 = reinterpret_cast<uint16_t*>(qa_s);
        const int quad = hh / 4, rr = hh % 4;
        const uint16_t hi = to_bf16(x);
        const uint16_t lo = to_bf16(x - bf16lo(hi));
        qa16[(((quad * 2 + 0) * 4 + rr) * DC) * 8 + i] = hi;
        qa16[(((quad * 2 + 1) * 4 + rr) * DC) * 8 + i] = lo;
      } else {
        qf_s[i][hh] = x * scale;
      }
    }
  }
  if (tid < G) teff_s[tid] = DENSE ? 0.f : tau_in - a.offset_a;
  for (int idx = tid; idx < NW * 64 * GQ; idx += NT) (&p_s[0][0])[idx] = 0.f;

  // The split's share of the list (the union's blocks, or every block when
  // dense): on the bf16 path the list's 64-token tiles s, s + S, s + 2 S, ...
  // (shares differ by at most one tile and each spreads over the whole list,
  // which measured faster than contiguous ranges); on the fp32 path the
  // contiguous range of whole blocks [lo, hi).
  int64_t UI;                // items (blocks) in the list
  if constexpr (DENSE) {
    UI = N;
  } else if constexpr (!uniform) {
    UI = pref[g.n_tiles] - pbase;   // the plan's scan holds the group's prefix
  } else {
    // exclusive prefix sum of the per-tile union counts, NT tiles at a time
    int carry = 0;
    for (int base = 0; base < g.n_tiles; base += NT) {
      const int t = base + tid;
      const int x = base == 0 ? tc0 : (t < g.n_tiles ? tc[t] : 0);
      const int incl = wave_incl_scan(x);
      if (lane == 63) wsum_s[w] = incl;
      __syncthreads();
      int woff = 0, tot = 0;
#pragma unroll
      for (int k = 0; k < NW; ++k) {
        woff += (k < w) ? wsum_s[k] : 0;
        tot += wsum_s[k];
      }
      if (t < g.n_tiles) pref_s[t] = carry + woff + incl - x;
      carry += tot;
      __syncthreads();
    }
    if (tid == 0) pref_s[g.n_tiles] = carry;
    UI = carry;
  }
  // top-1 rescue (App. "Top-1 Rescue, Tail Handling, and Kernel Validation"):
  // for each head, when no block of the window [0, Wn) is selected, the first of
  // the window's largest bounds (tiles in order, strict >, each tile's own first
  // largest) is attended as well.  Each distinct rescued block becomes one more
  // item of the list, after the union's, carrying the heads that rescued it (a
  // rescued head attends it only there, also when the block is in the union for
  // other heads, which then reads it once more).
  int jr_h = -1;                  // tid < G: head tid's rescued block, or -1
  uint32_t wb_rescued = 1u;
  if constexpr (!DENSE) {
    if (tid < G) {
      int jr = -1;
      if (a.c > 0 && Wn > 0) {
        bool any = false;
        float best = kNegInf;
        int arg = -1;
        for (int t = 0; t < nwt; ++t) {
          const int inf = rinfo_s[tid][t];
          if (inf == kRescueAny) {
            any = true;
          } else if (inf >= 0 && (arg < 0 || rbest_s[tid][t] > best)) {
            best = rbest_s[tid][t];
            arg = inf;
          }
        }
        if (!any) jr = arg;
      }
      resc_s[tid] = jr;
      jr_h = jr;
    }
    // whether the rescued block is in the union: for the union count only (the
    // last split writes it after streaming)
    if (tid < G && s == S - 1 && jr_h >= 0) wb_rescued = a.wbits[bg * kMaxRescueWindow + jr_h];
    if (s == 0 && tid == 0) a.plan[bg] = make_int2(first, S);
    __syncthreads();
    if (tid == 0) {
      int nb = 0;
      for (int h = 0; h < G; ++h) {
        const int j = resc_s[h];
        if (j < 0) continue;
        int k = 0;
        while (k < nb && rx_s[k][0] != j) ++k;
        if (k == nb) {
          rx_s[nb][0] = j;
          rx_s[nb][1] = 0;
          ++nb;
        }
        rx_s[k][1] |= 1 << h;
      }
      nrx_s = nb;
    }
    __syncthreads();
  }
  const int64_t UI_union = UI;
  if constexpr (!DENSE) UI += nrx_s;
  int64_t lo, hi;
  contiguous_share(UI, s, S, &lo, &hi);
  __syncthreads();

  const KVT* kb = reinterpret_cast<const KVT*>(a.k) + (int64_t)b * g.sb + (int64_t)gh * g.sh;
  const KVT* vb = reinterpret_cast<const KVT*>(a.v) + (int64_t)b * g.sb + (int64_t)gh * g.sh;
  const int64_t self_t = (!DENSE && a.self_ungated) ? T - 1 : -1;
  const bool use_lo = a.q_dtype == ETA_DT_F32;
  float m_[G], l_[G], acc[G][DPL];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m_[h] = kNegInf;
    l_[h] = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) acc[h][e] = 0.f;
  }
  auto attend = [&](int64_t t0, int nvalid, uint32_t bits) {
    if constexpr (BF)
      attend_bf16<D, G, DENSE>(kb, vb, g.st, t0, nvalid, bits, qa_s, use_lo, teff_s, p_s[w],
                               a.beta, scale, self_t, lane, m_, l_, acc);
    else
      attend_f32<D, G, DENSE>(kb, vb, g.st, t0, nvalid, bits, qf_s,
                              teff_s, reinterpret_cast<float (*)[G]>(p_s[w]), a.beta, self_t, lane,
                              m_, l_, acc);
  };
  constexpr uint32_t all_bits = (1u << G) - 1u;
  // The split's items are resolved (union slot -> block id -> head bits) in
  // chunks by all threads at once and kept in LDS, so a wavefront's K/V loads
  // never wait on those lookups.
  // list item -> (block id, head bits)
  auto resolve = [&](int64_t it, int32_t& jo, uint8_t& bo) {
    if constexpr (DENSE) {
      jo = (int32_t)it;
      bo = (uint8_t)all_bits;
    } else if (it >= UI_union) {        // rescued block: the heads that rescued it
      jo = rx_s[it - UI_union][0];
      bo = (uint8_t)rx_s[it - UI_union][1];
    } else {
      int tl, slot;
      resolve_item(pref, g.n_tiles, it + pbase, &tl, &slot);
      const uint32_t id = (uint32_t)a.ids[bg * g.ncap + (int64_t)tl * kScreenTile + slot];
      jo = (int32_t)(id & kIdMask);
      bo = (uint8_t)(id >> 24);
    }
  };
  if constexpr (BF) {
    // kItemChunk of the share's tiles at a time, resolved by all threads at once;
    // wavefront w takes the chunk's tiles w, w + NW, ... so the wavefronts finish
    // within one tile
    const int nt = strided_share(UI * SPB, s, S);
    for (int k0 = 0; k0 < nt; k0 += kItemChunk) {
      const int n = nt - k0 < kItemChunk ? nt - k0 : kItemChunk;
      if (tid < n) {
        const int64_t t = s + (int64_t)S * (k0 + tid);
        resolve(t / SPB, item_j[tid], item_bits[tid]);
        item_sub[tid] = (uint8_t)(t % SPB);
      }
      __syncthreads();
      const int nmine = n > w ? (n - w + NW - 1) / NW : 0;
      attend_bf16_stream<D, G, DENSE>(
          kb, vb, g.st, nmine,
          [&](int u) {
            const int x = w + NW * u;
            return (int64_t)item_j[x] * BS + 64 * item_sub[x];
          },
          [&](int u) { return (uint32_t)item_bits[w + NW * u]; }, qa_s, use_lo, teff_s, p_s[w],
          a.beta, scale, self_t, lane, m_, l_, acc);
      __syncthreads();
    }
  } else {
    for (int64_t base = lo; base < hi; base += kItemChunk) {
      const int n = (int)(hi - base < kItemChunk ? hi - base : kItemChunk);
      if (tid < n) resolve(base + tid, item_j[tid], item_bits[tid]);
      __syncthreads();
      for (int k = w; k < n; k += NW) attend((int64_t)item_j[k] * BS, BS, item_bits[k]);
      __syncthreads();
    }
  }
  if constexpr (!DENSE) {
    if (s == S - 1) {
      // the rescued blocks' mask bits, and (for the combine) each head's rescued
      // block and how many rescued blocks are outside the union
      if (tid < G) rxw_s[tid] = jr_h >= 0 ? (int)wb_rescued : 1;   // union bits at the rescued block
      __syncthreads();
      if (tid == 0) {
        int extra = 0;
        for (int k = 0; k < nrx_s; ++k) {
          int in_union = 0;
          for (int h = 0; h < G; ++h) in_union |= (resc_s[h] == rx_s[k][0] && rxw_s[h] != 0);
          extra += !in_union;
        }
        if (!single)
          a.extra_union[bg] = extra;
        else if (a.union_counts != nullptr)
          a.union_counts[bg] = (int32_t)(UI_union + extra);
      }
      if (tid < G) {
        if (!single) a.resc_out[hq0 + tid] = resc_s[tid];
        if (resc_s[tid] >= 0) a.mask[(hq0 + tid) * g.ncap + resc_s[tid]] = 1;
      }
    }
  }
  if (s == S - 1 && ntail > 0 && w == NW - 1) attend(N * BS, ntail, all_bits);

  // merge the four wavefront states
  if (lane == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) { mrg_ml[w][h][0] = m_[h]; mrg_ml[w][h][1] = l_[h]; }
  }
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < DPL; ++e) mrg_acc[w][h][lane * DPL + e] = acc[h][e];
  __syncthreads();
  for (int idx = tid; idx < G * D; idx += NT) {
    const int h = idx / D, i = idx % D;
    float ms = kNegInf;
#pragma unroll
    for (int k = 0; k < NW; ++k) ms = fmaxf(ms, mrg_ml[k][h][0]);
    float L = 0.f, o = 0.f;
    if (ms != kNegInf) {
#pragma unroll
      for (int k = 0; k < NW; ++k) {
        const float mk = mrg_ml[k][h][0];
        if (mk == kNegInf) continue;
        const float wk = __expf(mk - ms);
        L = fmaf(mrg_ml[k][h][1], wk, L);
        o = fmaf(mrg_acc[k][h][i], wk, o);
      }
    }
    if (single) {          // the combine's result for one partial: acc / l
      store_out(a.out, a.q_dtype, (hq0 + h) * D + i, L > 0.f ? o / L : 0.f);
    } else {
      const int64_t pidx = (int64_t)(first + s) * G + h;
      a.part_acc[pidx * D + i] = o;
      if (i == 0) a.part_ml[pidx] = make_float2(ms, L);
    }
  }
  if constexpr (!DENSE) {
    if (single && a.counts != nullptr) {
      // attended tokens per head: its selected blocks (tile counts), its
      // rescued block, the tail
      for (int h = w; h < G; h += NW) {
        int cnt = 0;
        for (int t = lane; t < g.n_tiles; t += 64) cnt += a.head_cnt[(hq0 + h) * g.n_tiles + t];
#pragma unroll
        for (int o2 = 32; o2 > 0; o2 >>= 1) cnt += __shfl_xor(cnt, o2, 64);
        if (lane == 0)
          a.counts[hq0 + h] = (int32_t)(((int64_t)cnt + (resc_s[h] >= 0 ? 1 : 0)) * BS + ntail);
      }
    }
  }
}

// ---------------------------------------------------------------- calibration
//
// Offline density-matched calibration.  calib_kernel: one workgroup per
// (query head, sequence); wavefront w takes the 16-query groups w, w + 4, ...
// and, for each, the 16-key blocks 0 .. group (the causal triangle).  Scores
// come from v_mfma_f32_16x16x32_bf16 in the standard layout: A = 16 query rows
// x 32 dims, B = 32 dims x 16 keys, so lane l gets the scores of queries
// 4 (l >> 4) + i of the group and key l & 15 of the block.  Each causal score
// adds its step's weight round(2^40 / (t + 1)) to an LDS histogram with a
// 64-bit integer atomic; the lane's gate sum sigmoid(beta (S - tau_t)) / (t + 1)
// accumulates in fp64 in a fixed order and is added once, rounded to the same
// fixed point.  Integer sums make the result independent of the adds' order.
// calib_solve_kernel: one workgroup per head, fp64 bisection of the
// histogram's density function with fixed-order block reductions.

constexpr int kCalibMaxBins = 4096;
constexpr double kCalibUnit = 1099511627776.0;   // 2^40

struct CalibArgs {
  const uint16_t* q;
  const uint16_t* k;
  const float* tau;
  unsigned long long* hist;
  unsigned long long* dens;
  int Hq, Hkv, T, nb;
  float beta, lo, inv_w;
};

template <int D>
__global__ __launch_bounds__(256) void calib_kernel(CalibArgs a) {
  constexpr int KC = D / 32;                      // 32-dim chunks
  __shared__ unsigned long long hist_s[kCalibMaxBins];
  const int h = blockIdx.x, x = blockIdx.y, tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int G = a.Hq / a.Hkv;
  for (int b = tid; b < a.nb; b += 256) hist_s[b] = 0ull;
  __syncthreads();
  const uint16_t* qh = a.q + (((int64_t)x * a.Hq + h) * a.T) * D;
  const uint16_t* kh = a.k + (((int64_t)x * a.Hkv + h / G) * a.T) * D;
  const float* tauh = a.tau + ((int64_t)x * a.Hq + h) * a.T;
  const float scale = 1.0f / sqrtf((float)D);
  const int ngroups = (a.T + 15) / 16;
  const int r16 = lane & 15, g4 = lane >> 4;
  double dens = 0.0;
  for (int qg = w; qg < ngroups; qg += 4) {
    // A: query row 16 qg + r16, dims 32 kc + 8 g4 .. + 7 (rows past T read row T - 1)
    const int qr = min(16 * qg + r16, a.T - 1);
    bf16x8 qa[KC];
#pragma unroll
    for (int kc = 0; kc < KC; ++kc)
      qa[kc] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(qh + (int64_t)qr * D + 32 * kc + 8 * g4));
    // this lane's output rows: steps t_i = 16 qg + 4 g4 + i
    int t_i[4];
    float tau_i[4], invt_i[4];
    unsigned long long wt_i[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      t_i[i] = 16 * qg + 4 * g4 + i;
      const int tc = min(t_i[i], a.T - 1);
      tau_i[i] = tauh[tc];
      invt_i[i] = 1.0f / (float)(t_i[i] + 1);
      wt_i[i] = (unsigned long long)llrint(kCalibUnit / (double)(t_i[i] + 1));
    }
    for (int kb = 0; kb <= qg; ++kb) {
      const int kr = min(16 * kb + r16, a.T - 1);
      bf16x8 kk[KC];
#pragma unroll
      for (int kc = 0; kc < KC; ++kc)
        kk[kc] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(kh + (int64_t)kr * D + 32 * kc + 8 * g4));
      f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kc = 0; kc < KC; ++kc) c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[kc], kk[kc], c, 0, 0, 0);
      const int s_idx = 16 * kb + r16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (s_idx <= t_i[i] && t_i[i] < a.T) {
          const float S = c[i] * scale;
          float f = floorf((S - a.lo) * a.inv_w);
          f = f >= 0.f ? f : 0.f;        // also NaN
          const int bin = f < (float)a.nb ? (int)f : a.nb - 1;
          atomicAdd(&hist_s[bin], wt_i[i]);
          const float gate = 1.0f / (1.0f + __expf(-a.beta * (S - tau_i[i])));
          dens += (double)(gate * invt_i[i]);
        }
      }
    }
  }
  // the lane's gate sum in fixed point; integer wavefront sum; one global add
  unsigned long long dv = (unsigned long long)llrint(dens * kCalibUnit);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) dv += __shfl_xor(dv, o, 64);
  if (lane == 0) atomicAdd(&a.dens[h], dv);
  __syncthreads();
  for (int b = tid; b < a.nb; b += 256) {
    const unsigned long long v = hist_s[b];
    if (v != 0ull) atomicAdd(&a.hist[(int64_t)h * a.nb + b], v);
  }
}

__device__ __forceinline__ double sigmoid_f64(double x) {
  if (x >= 0.0) return 1.0 / (1.0 + exp(-x));
  const double e = exp(x);
  return e / (1.0 + e);
}

__device__ __forceinline__ double block_sum_f64(double x, double* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  if (lane == 0) red[w] = x;
  __syncthreads();
  const double r = ((red[0] + red[1]) + red[2]) + red[3];
  __syncthreads();
  return r;
}

struct CalibSolveArgs {
  const unsigned long long* hist;
  const unsigned long long* dens;
  float* c_out;
  double* target_out;
  int nb;
  double beta, lo, hi;
};

#if ETA_PART == 0
__global__ __launch_bounds__(256) void calib_solve_kernel(CalibSolveArgs a) {
  constexpr int PER = kCalibMaxBins / 256;
  __shared__ double red[4];
  const int h = blockIdx.x, tid = threadIdx.x;
  const double w = (a.hi - a.lo) / (double)a.nb;
  double hb[PER], sb[PER];
  double tot = 0.0;
#pragma unroll
  for (int r = 0; r < PER; ++r) {
    const int b = tid + 256 * r;
    hb[r] = b < a.nb ? (double)a.hist[(int64_t)h * a.nb + b] : 0.0;
    sb[r] = a.lo + ((double)b + 0.5) * w;
    tot += hb[r];
  }
  tot = block_sum_f64(tot, red);
  const double target = (double)a.dens[h] / tot;
  double lo = a.lo - 60.0 / a.beta, hi = a.hi + 60.0 / a.beta;
  for (int it = 0; it < 2048; ++it) {
    const double m = 0.5 * (lo + hi);
    if (m <= lo || m >= hi) break;
    double g = 0.0;
#pragma unroll
    for (int r = 0; r < PER; ++r) g += hb[r] * sigmoid_f64(a.beta * (sb[r] - m));
    g = block_sum_f64(g, red) / tot;
    if (g > target) lo = m; else hi = m;
  }
  if (tid == 0) {
    a.c_out[h] = tot > 0.0 ? (float)(0.5 * (lo + hi)) : __builtin_nanf("");
    if (a.target_out != nullptr) a.target_out[h] = tot > 0.0 ? target : __builtin_nan("");
  }
}
#endif

// ---------------------------------------------------------------- combine

struct CombineArgs {
  const float2* part_ml;     // [splits][G]
  const float* part_acc;     // [splits][G][D]
  const int32_t* head_cnt;
  const int32_t* tile_cnt;
  const int32_t* seq_lens;
  const int32_t* resc_out;   // rescued block per head or -1 (nullptr: dense)
  const int32_t* extra_union;
  const int2* plan;          // (first split, splits) per group; nullptr: uniform S
  int32_t* counts;
  int32_t* union_counts;
  void* out;
  Geom g;
  int q_dtype;
  int S;                     // uniform splits per group (plan == nullptr)
};

// One workgroup of 512 threads per (sequence, query head).  Thread (i, part)
// owns head dimension i and the splits s = part, part + P, ... (P = 512 / D):
// it issues the loads of its splits' maxima and accumulators together, the
// workgroup takes the largest maximum, and each thread adds its weighted
// accumulators exp(m_s - m) acc_s[i] (the part-0 threads also the weighted
// sums l_s); the P partial sums are then added in order.  (512 threads: 0.5 us
// faster than 1024 at 64 splits, fewer wavefronts in each reduction; 256 left
// 32 splits per thread and was no faster.)
constexpr int kCombThreads = 512;
constexpr int kCombPrefetch = 16;

__device__ __forceinline__ float block_reduce(float x, bool is_max, float* red) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  x = is_max ? wave_max(x) : wave_sum(x);
  if (lane == 0) red[w] = x;
  __syncthreads();
  float r = red[0];
  for (int k = 1; k < (int)(blockDim.x >> 6); ++k) r = is_max ? fmaxf(r, red[k]) : r + red[k];
  __syncthreads();
  return r;
}

template <int D>
__global__ __launch_bounds__(kCombThreads) void combine_kernel(CombineArgs a) {
  constexpr int P = kCombThreads / D;
  __shared__ float red[kCombThreads];
  __shared__ float lred[P];
  const Geom& g = a.g;
  const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int i = tid % D, part = tid / D;
  const int64_t row = (int64_t)b * g.Hq + h;
  const int64_t bg = (int64_t)b * g.Hkv + h / g.G;
  const int hh = h % g.G;
  // per-head selected blocks: wavefront 0 sums the head's tile counts; the
  // union blocks of the (sequence, kv head): wavefront 1 of the group's first
  // head sums the union's tile counts.  The first 64 of each are loaded here
  // (every thread, from clamped indexes, so no load waits inside a branch or
  // a loop) together with the rescue results, the sequence length and the
  // group's split range, and summed at the end (row shifts on the vector ALUs);
  // tiles past 64 are read there.
  const int lt = tid & 63, ti = lt < g.n_tiles ? lt : 0;
  const bool do_cnt = a.counts != nullptr && tid < 64;
  const bool do_union = a.union_counts != nullptr && hh == 0 && tid >= 64 && tid < 128;
  int cnt = a.counts != nullptr ? a.head_cnt[row * g.n_tiles + ti] : 0;
  int ucnt = a.union_counts != nullptr ? a.tile_cnt[bg * g.n_tiles + ti] : 0;
  const int rescued = (a.resc_out != nullptr && tid == 0) ? a.resc_out[row] : -1;
  const int32_t len_raw = a.seq_lens[b];      // for the attended-token count
  const int extra = (a.extra_union != nullptr && tid == 64 && do_union) ? a.extra_union[bg] : 0;
  int first = (int)bg * a.S, S = a.S;
  if (a.plan != nullptr) {
    const int2 pl = a.plan[bg];
    first = pl.x;
    S = pl.y;
  }
  // split s's partial of this head: (first + s) G + hh
  const float2* ml = a.part_ml + (int64_t)first * g.G + hh;
  const float* accp = a.part_acc + ((int64_t)first * g.G + hh) * D + i;
  const int64_t st = g.G;          // partials between consecutive splits
  float2 mv[kCombPrefetch];
  float av[kCombPrefetch];
  float mloc = kNegInf;
#pragma unroll
  for (int k = 0; k < kCombPrefetch; ++k) {
    const int sidx = part + P * k;
    const bool in = sidx < S;
    mv[k] = in ? ml[sidx * st] : make_float2(kNegInf, 0.f);
    av[k] = in ? accp[sidx * st * D] : 0.f;
    mloc = fmaxf(mloc, mv[k].x);
  }
  // splits past the prefetched ones (more than 16 per thread): unrolled so that
  // eight loads are in flight at a time instead of one round trip per split
#pragma unroll 8
  for (int sidx = part + P * kCombPrefetch; sidx < S; sidx += P) mloc = fmaxf(mloc, ml[sidx * st].x);
  const float ms = block_reduce(mloc, true, red);
  float o = 0.f, L = 0.f;
  if (ms != kNegInf) {
#pragma unroll
    for (int k = 0; k < kCombPrefetch; ++k) {
      const float wk = mv[k].x == kNegInf ? 0.f : __expf(mv[k].x - ms);
      o = fmaf(wk, av[k], o);
      L = fmaf(mv[k].y, wk, L);
    }
#pragma unroll 8
    for (int sidx = part + P * kCombPrefetch; sidx < S; sidx += P) {
      const float2 e = ml[sidx * st];
      const float wk = e.x == kNegInf ? 0.f : __expf(e.x - ms);
      o = fmaf(wk, accp[sidx * st * D], o);
      L = fmaf(e.y, wk, L);
    }
  }
  red[tid] = o;
  if (i == 0) lred[part] = L;
  __syncthreads();
  if (tid < D) {
    float x = 0.f, Lt = 0.f;
#pragma unroll
    for (int p = 0; p < P; ++p) {
      x += red[p * D + tid];
      Lt += lred[p];
    }
    store_out(a.out, a.q_dtype, row * D + tid, Lt > 0.f ? x / Lt : 0.f);
  }
  if (do_cnt) {
    cnt = lt < g.n_tiles ? cnt : 0;
    for (int t = lt + 64; t < g.n_tiles; t += 64) cnt += a.head_cnt[row * g.n_tiles + t];
    cnt = __builtin_amdgcn_readlane(wave_incl_scan(cnt), 63);
    if (tid == 0) {
      const int64_t T = len_raw < 0 ? 0 : (len_raw > g.cap ? g.cap : (int64_t)len_raw);
      const int64_t N = T / g.BS;
      a.counts[row] = (int32_t)(((int64_t)cnt + (rescued >= 0 ? 1 : 0)) * g.BS + (T - N * g.BS));
    }
  }
  if (do_union) {
    ucnt = lt < g.n_tiles ? ucnt : 0;
    for (int t = lt + 64; t < g.n_tiles; t += 64) ucnt += a.tile_cnt[bg * g.n_tiles + t];
    ucnt = __builtin_amdgcn_readlane(wave_incl_scan(ucnt), 63);
    if (tid == 64) a.union_counts[bg] = ucnt + extra;
  }
}

}  // namespace

// ---------------------------------------------------------------- launchers

// Split decode on one cache type (defined in object 1 for bf16, 2 for fp32).
template <bool DENSE, typename KVT>
void launch_split_kv(const Geom& g, const SplitPlan& pl, const SplitArgs& sp, hipStream_t stream);

#if ETA_PART == 1 || ETA_PART == 2
template <bool DENSE, typename KVT>
void launch_split_kv(const Geom& g, const SplitPlan& pl, const SplitArgs& sp, hipStream_t stream) {
  const dim3 grid = pl.S > 0 ? dim3(pl.S, g.Hkv, g.B) : dim3(pl.W);
#define ETA_SPL(D_, BS_, G_)                                                                    \
  if (g.D == D_ && g.BS == BS_ && g.G == G_) {                                                  \
    if (DENSE || pl.S > 0)                                                                      \
      hipLaunchKernelGGL((split_kernel<D_, BS_, G_, KVT, DENSE, false>), grid, dim3(64 * kSplitWaves), 0, \
                         stream, sp);                                                           \
    else                                                                                        \
      hipLaunchKernelGGL((split_kernel<D_, BS_, G_, KVT, DENSE, !DENSE>), grid, dim3(64 * kSplitWaves), 0, \
                         stream, sp);                                                           \
  }
#define ETA_SPL_G(D_, BS_) ETA_SPL(D_, BS_, 1) ETA_SPL(D_, BS_, 2) ETA_SPL(D_, BS_, 4) ETA_SPL(D_, BS_, 8)
  ETA_SPL_G(64, 64) ETA_SPL_G(64, 128) ETA_SPL_G(128, 64) ETA_SPL_G(128, 128)
#undef ETA_SPL_G
#undef ETA_SPL
}
#if ETA_PART == 1
template void launch_split_kv<false, uint16_t>(const Geom&, const SplitPlan&, const SplitArgs&, hipStream_t);
template void launch_split_kv<true, uint16_t>(const Geom&, const SplitPlan&, const SplitArgs&, hipStream_t);
#else
template void launch_split_kv<false, float>(const Geom&, const SplitPlan&, const SplitArgs&, hipStream_t);
template void launch_split_kv<true, float>(const Geom&, const SplitPlan&, const SplitArgs&, hipStream_t);
#endif
#endif

#if ETA_PART == 0

hipError_t launch_summaries(const Geom& g, const void* k, const int32_t* seq_lens,
                            const int32_t* prev_lens, int max_new_blocks, int sub_block,
                            const eta_summary_t& s, hipStream_t stream, LaunchHook hook) {
  const int64_t nblk = prev_lens != nullptr ? max_new_blocks : g.cap / g.BS;
  if (nblk <= 0) return hipSuccess;
  dim3 grid((unsigned)((nblk + kSumBlocks - 1) / kSumBlocks), g.Hkv, g.B);
  int sub_log2 = 0;
  while (sub_block > 0 && (1 << sub_log2) < sub_block) ++sub_log2;
  const int max_new = prev_lens != nullptr ? max_new_blocks : 0;
  return with_hook(hook, ETA_KERNEL_SUMMARIES, stream, [&] {
#define ETA_SUM(D_, BS_, T_)                                                                    \
  if (g.D == D_ && g.BS == BS_) {                                                               \
    if (sub_block > 0)                                                                          \
      hipLaunchKernelGGL((summaries_kernel<D_, BS_, T_, true>), grid, dim3(256), 0, stream,     \
                         reinterpret_cast<const T_*>(k), g, seq_lens, prev_lens, max_new,       \
                         sub_log2, s.mu, s.sigma, s.max_norm);                                  \
    else                                                                                        \
      hipLaunchKernelGGL((summaries_kernel<D_, BS_, T_, false>), grid, dim3(256), 0, stream,    \
                         reinterpret_cast<const T_*>(k), g, seq_lens, prev_lens, max_new,       \
                         sub_log2, s.mu, s.sigma, s.max_norm);                                  \
  }
    if (g.kv_dtype == ETA_DT_F32) {
      ETA_SUM(64, 64, float) ETA_SUM(64, 128, float) ETA_SUM(128, 64, float) ETA_SUM(128, 128, float)
    } else {
      ETA_SUM(64, 64, uint16_t) ETA_SUM(64, 128, uint16_t) ETA_SUM(128, 64, uint16_t)
      ETA_SUM(128, 128, uint16_t)
    }
#undef ETA_SUM
  });
}

hipError_t launch_predict(int B, int Hq, int D, int q_dtype, const void* q, const float* W,
                          const float* bias, float* tau, hipStream_t stream, LaunchHook hook) {
  return with_hook(hook, ETA_KERNEL_PREDICT, stream, [&] {
    hipLaunchKernelGGL(predict_kernel, dim3(B, (Hq + kPredCols - 1) / kPredCols), dim3(kPredThreads),
                       0, stream, q, q_dtype, W, bias, tau, Hq, D);
  });
}

namespace {

template <bool BOUNDS_ONLY>
void launch_screen_impl(const Geom& g, const ScreenArgs& sa, hipStream_t stream) {
  dim3 grid(g.n_tiles, g.Hkv, g.B);
  // four-record loads need rows that start on a multiple of 4 records
  const bool vec = g.ncap >= 4 && (g.ncap & 3) == 0;
#define ETA_SCR_T(D_, G_, ST_)                                                                  \
  if (vec)                                                                                      \
    hipLaunchKernelGGL((screen_kernel<D_, G_, BOUNDS_ONLY, ST_, true>), grid,                   \
                       dim3(kScreenThreads), 0, stream, sa);                                    \
  else                                                                                          \
    hipLaunchKernelGGL((screen_kernel<D_, G_, BOUNDS_ONLY, ST_, false>), grid,                  \
                       dim3(kScreenThreads), 0, stream, sa);
#define ETA_SCR(D_, G_)                                                                         \
  if (g.D == D_ && g.G == G_) {                                                                 \
    if (g.stat_dtype == ETA_DT_F16) {                                                           \
      ETA_SCR_T(D_, G_, _Float16)                                                               \
    } else if (g.stat_dtype == ETA_DT_FP8) {                                                    \
      ETA_SCR_T(D_, G_, uint8_t)                                                                \
    } else {                                                                                    \
      ETA_SCR_T(D_, G_, float)                                                                  \
    }                                                                                           \
  }
  ETA_SCR(64, 1) ETA_SCR(64, 2) ETA_SCR(64, 4) ETA_SCR(64, 8)
  ETA_SCR(128, 1) ETA_SCR(128, 2) ETA_SCR(128, 4) ETA_SCR(128, 8)
#undef ETA_SCR
#undef ETA_SCR_T
}

template <bool DENSE>
void launch_split_impl(const Geom& g, const SplitPlan& pl, const SplitArgs& sp, hipStream_t stream) {
  if (g.kv_dtype == ETA_DT_F32)
    launch_split_kv<DENSE, float>(g, pl, sp, stream);
  else
    launch_split_kv<DENSE, uint16_t>(g, pl, sp, stream);
}

void launch_combine_impl(const Geom& g, const CombineArgs& ca, hipStream_t stream) {
  dim3 grid(g.Hq, g.B);
  if (g.D == 64) hipLaunchKernelGGL(combine_kernel<64>, grid, dim3(kCombThreads), 0, stream, ca);
  if (g.D == 128) hipLaunchKernelGGL(combine_kernel<128>, grid, dim3(kCombThreads), 0, stream, ca);
}

}  // namespace

// L2 bytes of W that the fused predictor may re-read per step (see launch_decode)
constexpr int64_t kFusedPredictMaxBytes = 64ll << 20;

hipError_t launch_decode(const Geom& g, const DecodeCfg& c, int q_dtype, const void* q,
                         const void* k, const void* v, const int32_t* seq_lens,
                         const eta_summary_t& s, const float* tau, const float* W,
                         const float* bias, float* tau_out, void* out, uint8_t* mask,
                         int32_t* counts, int32_t* union_counts, const DecodeWs& ws,
                         hipStream_t stream, LaunchHook hook) {
  const bool predict = tau == nullptr;
  // The fused predictor reads its group's G rows of W in every screening
  // workgroup: B Hkv n_tiles Hq D G 4 bytes of L2 reads per step.  Past
  // kFusedPredictMaxBytes the thresholds are predicted once per step by
  // predict_kernel into the workspace (the same arithmetic in the same order,
  // so the thresholds are bit-identical) and screening reads them.
  const bool separate = predict && W != nullptr &&
                        (int64_t)g.B * g.Hkv * g.n_tiles * g.Hq * g.D * g.G * 4 > kFusedPredictMaxBytes;
  if (separate) {
    const hipError_t e0 = launch_predict(g.B, g.Hq, g.D, q_dtype, q, W, bias, ws.tau, stream, hook);
    if (e0 != hipSuccess) return e0;
  }
  ScreenArgs sa{q, seq_lens, separate ? ws.tau : tau, W, bias, ws.tau, tau_out, s.mu, s.sigma,
                s.max_norm, mask, ws.ids, ws.tile_cnt, ws.head_cnt, nullptr, ws.resc_best,
                ws.resc_info, ws.wbits, g, q_dtype, (predict && !separate) ? 1 : 0, c.z,
                c.offset_a, c.rescue_window, c.lwb, c.screen_all};
  hipError_t e = with_hook(hook, ETA_KERNEL_SCREEN, stream,
                           [&] { launch_screen_impl<false>(g, sa, stream); });
  if (e != hipSuccess) return e;
  SplitArgs sp{q, k, v, seq_lens, predict ? ws.tau : tau, ws.ids, ws.tile_cnt, ws.part_ml,
               ws.part_acc, ws.resc_best, ws.resc_info, ws.wbits, mask, ws.resc_out,
               ws.extra_union, ws.plan, ws.head_cnt, out, counts, union_counts, g, q_dtype,
               c.beta, c.offset_a, c.self_ungated, c.rescue_window};
  e = with_hook(hook, ETA_KERNEL_SPLIT_DECODE, stream,
                [&] { launch_split_impl<false>(g, c.plan, sp, stream); });
  if (e != hipSuccess) return e;
  if (c.plan.S == 1) return hipSuccess;     // one split per group wrote the results
  CombineArgs ca{ws.part_ml, ws.part_acc, ws.head_cnt, ws.tile_cnt, seq_lens, ws.resc_out,
                 ws.extra_union, c.plan.S > 0 ? nullptr : ws.plan, counts, union_counts, out, g,
                 q_dtype, c.plan.S};
  return with_hook(hook, ETA_KERNEL_COMBINE, stream, [&] { launch_combine_impl(g, ca, stream); });
}

hipError_t launch_bounds(const Geom& g, int q_dtype, const void* q, const int32_t* seq_lens,
                         const eta_summary_t& s, float z, float* bounds, hipStream_t stream,
                         LaunchHook hook) {
  ScreenArgs sa{q, seq_lens, nullptr, nullptr, nullptr, nullptr, nullptr, s.mu, s.sigma,
                s.max_norm, nullptr, nullptr, nullptr, nullptr, bounds, nullptr, nullptr, nullptr,
                g, q_dtype, 0, z, 0.f, 0, 0, 0};
  return with_hook(hook, ETA_KERNEL_BOUNDS, stream,
                   [&] { launch_screen_impl<true>(g, sa, stream); });
}

hipError_t launch_calib(const eta_calib_desc_t& cd, const void* q, const void* k, const float* tau,
                        const eta_calib_state_t& st, hipStream_t stream, LaunchHook hook) {
  CalibArgs ca{reinterpret_cast<const uint16_t*>(q), reinterpret_cast<const uint16_t*>(k), tau,
               reinterpret_cast<unsigned long long*>(st.hist),
               reinterpret_cast<unsigned long long*>(st.density), cd.num_q_heads, cd.num_kv_heads,
               cd.seq_len, cd.num_bins, cd.beta, cd.lo,
               (float)((double)cd.num_bins / ((double)cd.hi - (double)cd.lo))};
  dim3 grid(cd.num_q_heads, cd.num_seqs);
  return with_hook(hook, ETA_KERNEL_CALIB_ACCUMULATE, stream, [&] {
    if (cd.head_dim == 64) hipLaunchKernelGGL(calib_kernel<64>, grid, dim3(256), 0, stream, ca);
    if (cd.head_dim == 128) hipLaunchKernelGGL(calib_kernel<128>, grid, dim3(256), 0, stream, ca);
  });
}

hipError_t launch_calib_solve(const eta_calib_desc_t& cd, const eta_calib_state_t& st, float* c_out,
                              double* target_out, hipStream_t stream, LaunchHook hook) {
  CalibSolveArgs sa{reinterpret_cast<const unsigned long long*>(st.hist),
                    reinterpret_cast<const unsigned long long*>(st.density), c_out, target_out,
                    cd.num_bins, (double)cd.beta, (double)cd.lo, (double)cd.hi};
  return with_hook(hook, ETA_KERNEL_CALIB_SOLVE, stream, [&] {
    hipLaunchKernelGGL(calib_solve_kernel, dim3(cd.num_q_heads), dim3(256), 0, stream, sa);
  });
}

hipError_t launch_dense(const Geom& g, int S, int q_dtype, const void* q, const void* k,
                        const void* v, const int32_t* seq_lens, void* out, const DecodeWs& ws,
                        hipStream_t stream, LaunchHook hook) {
  SplitArgs sp{q, k, v, seq_lens, nullptr, nullptr, nullptr, ws.part_ml, ws.part_acc,
               nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, out,
               nullptr, nullptr, g, q_dtype, 0.f, 0.f, 0, 0};
  hipError_t e = with_hook(hook, ETA_KERNEL_DENSE_SPLIT, stream,
                           [&] { launch_split_impl<true>(g, SplitPlan{S, S * g.B * g.Hkv}, sp, stream); });
  if (e != hipSuccess || S == 1) return e;     // one split per group wrote the output
  CombineArgs ca{ws.part_ml, ws.part_acc, nullptr, nullptr, seq_lens, nullptr, nullptr, nullptr,
                 nullptr, nullptr, out, g, q_dtype, S};
  return with_hook(hook, ETA_KERNEL_DENSE_COMBINE, stream,
                   [&] { launch_combine_impl(g, ca, stream); });
}

// ---------------------------------------------------------------- library scratch
//
// Workspace of eta_decode_predicted_noalloc: a file-scope device array (each GPU
// the library runs on holds its own copy, at its own address, until the
// process ends).  Host code never uses the array's name as an address: the
// device address of each GPU's copy is looked up once, with that GPU current,
// and kept.

__device__ __align__(256) unsigned char scratch[kScratchBytes];

hipError_t scratch_address(hipStream_t stream, void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  hipDevice_t dev = 0;
  hipError_t e = hipStreamGetDevice(stream, &dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(mu);
  if (addr[dev] == nullptr) {
    int cur = 0;
    if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) {
      const hipError_t e2 = hipSetDevice(cur);
      if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}

#endif  // ETA_PART == 0

}  // namespace eta
