// Gated prefill / training forward of libeta for gfx950 (CDNA4, wave64):
// causal attention over gated scores, with the per-row gate sums R and the
// log-sum-exp L (paper: "Elastic Threshold Attention", App. "Hardware-Aligned
// Forward Kernel", Alg. fwd_kernel).  fp32 accumulation, bf16 operands.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "eta_device.h"
#include "eta_internal.h"

namespace eta {
namespace {

// ---------------------------------------------------------------- gated prefill forward
//
// The training / prefill forward (App. "Hardware-Aligned Forward Kernel"):
// causal attention over gated scores S~ = S sigma(beta (S - tau_i)) (or the
// additive S + C sigma - C), diagonal ungated, with the gate row sums R and the
// log-sum-exp L.  One workgroup per (64-query block, query head, sequence),
// longest blocks first; wavefront w owns query rows 16 w .. 16 w + 15.  K and
// V blocks of 64 keys go straight from global memory into one of two LDS
// buffers (global_load_lds, 16 bytes per lane, no staging registers) while the
// other buffer is in use; rows are unpadded with their 16-byte chunks XOR
// swizzled by row, so the column reads of all 16 rows hit distinct banks.  One
// barrier per block.  Everything is computed transposed so that
// each lane owns one query row: S^T = K Q^T on v_mfma_f32_16x16x32_bf16 (A = 16
// keys x 32 dims from LDS, B = 32 dims x 16 queries from registers) gives lane l
// the scores of query l & 15 against keys 4 (l >> 4) + i of each 16-key
// quarter; the gate, mask and online softmax are per lane, with the four lane
// groups of a row combined by row / half-wave swaps; O^T += V^T P^T takes B =
// the lane's own gated weights (bf16), the contraction over keys permuted
// consistently on both sides, and A = V^T from two LDS transpose reads
// (ds_read_b64_tr_b16) of the row-major V tile.  fp32 accumulators.

constexpr int kPfQ = 128;    // query rows per workgroup (32 per wavefront)
constexpr int kPfK = 64;     // keys per block

struct PrefillArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const float* tau;
  const int32_t* seq_lens;
  uint16_t* out;
  float* R;
  float* L;
  int Hq, Hkv, T;
  float beta, C;
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

// lanes l, l ^ 16, l ^ 32, l ^ 48 hold the same query row
__device__ __forceinline__ float row4_max(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float row4_sum(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Swizzled 16-byte chunk of (row, chunk) in an unpadded LDS tile of rows of D
// bf16: rows sharing a 256-byte bank line are XORed with different values.
template <int D>
__device__ __forceinline__ int pf_chunk(int row, int chunk) {
  constexpr int CPR = D / 8, RPL = 128 / D;   // chunks per row, rows per 256 bytes
  return chunk ^ ((row / RPL) & (CPR - 1));
}

template <int D, bool ADD>
__global__ __launch_bounds__(256, 2) void prefill_kernel(PrefillArgs a) {
  constexpr int KC = D / 32;             // 32-dim chunks (score contraction)
  constexpr int DB = D / 16;             // 16-dim output blocks
  constexpr int CPR = D / 8;             // 16-byte chunks per K / V row
  constexpr int NI = kPfK * CPR / 256;   // DMA slots per thread per block and tensor
  __shared__ __attribute__((aligned(16))) uint16_t k_s[2][kPfK * D];
  __shared__ __attribute__((aligned(16))) uint16_t v_s[2][kPfK * D];

  const int nqb = (a.T + kPfQ - 1) / kPfQ;
  const int qblk = nqb - 1 - (int)blockIdx.x;        // longest causal ranges first
  const int h = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
  const int lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g4 = lane >> 4;
  const int G = a.Hq / a.Hkv;
  const int Tb = (int)clamp_len(a.seq_lens, b, a.T);
  const int64_t qrow0 = ((int64_t)b * a.Hq + h) * a.T;
  const uint16_t* kh = a.k + (((int64_t)b * a.Hkv + h / G) * a.T) * D;
  const uint16_t* vh = a.v + (((int64_t)b * a.Hkv + h / G) * a.T) * D;
  // Softmax and gate in base-2 units (S' = S log2 e): exp(S~ - m) = 2^(S~' - m') and
  // sigmoid(beta (S - tau)) = 1 / (1 + 2^(-beta (S' - tau'))).  With c the raw
  // product q.k and s2 = log2(e) / sqrt(d): S' = s2 c, and the lane keeps
  // gs = s2 sigmoid = 1 / ((1 + e) / s2), so the gated score is c gs (no separate
  // scaling) and R = (sum of gs) / s2.
  constexpr float kLog2e = 1.4426950408889634f;
  const float s2 = kLog2e / sqrtf((float)D), is2 = 1.0f / s2;
  const float nbs = -a.beta * s2;
  const float C2 = a.C * kLog2e, C2is = C2 * is2;

  // the wavefront's rows: t[hh] = base + 32 w + 16 hh + (lane & 15); B operands
  // of its queries (dims 32 kc + 8 g4 .. + 7)
  const int wrow0 = qblk * kPfQ + 32 * w;
  int t[2];
  float btau2[2], m_i[2], l_i[2], r_i[2];
  u32x4 qb[2][KC];
  f32x4 acc[2][DB];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    t[hh] = wrow0 + 16 * hh + r16;
    const int tq = min(t[hh], a.T - 1);
#pragma unroll
    for (int kc = 0; kc < KC; ++kc)
      qb[hh][kc] = *reinterpret_cast<const u32x4*>(a.q + (qrow0 + tq) * D + 32 * kc + 8 * g4);
    btau2[hh] = a.beta * a.tau[qrow0 + tq] * kLog2e;
    m_i[hh] = 0.f;    // reference maximum; set by the first block
    l_i[hh] = 0.f;    // this lane's share of the row's weight sum
    r_i[hh] = 0.f;    // this lane's share of the row's gate sum (times s2)
#pragma unroll
    for (int db = 0; db < DB; ++db) acc[hh][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // transpose reads of V: the lane provides key 4 g4 + (r16 >> 2) (+16 for keys
  // 16..31 of a 32-key chunk) and dims 4 (lane & 3) .. + 3 of a 16-dim block
  const int vt_row = 4 * g4 + (r16 >> 2), vt_c = lane & 3;

  // Key blocks of the workgroup and of this wavefront.  The wavefront's last
  // block holds its diagonal (or the sequence's end) and is the only one that
  // needs a mask; the blocks after it, up to the workgroup's last, it skips.
  const int last_row = min(qblk * kPfQ + kPfQ, Tb) - 1;
  const int nkb = last_row >= 0 ? last_row / kPfK + 1 : 0;
  const int nkb_w = wrow0 < Tb ? (min(wrow0 + 32, Tb) - 1) / kPfK + 1 : 0;

  // DMA: LDS slot u = 256 j + tid (16 bytes, in order) of a block holds row
  // u / CPR, physical chunk u % CPR, i.e. the global chunk that the swizzle maps
  // there.  Slot j of a thread is row RPJ j + tid / CPR, and its swizzle term
  // (row / (128 / D)) mod CPR does not depend on j, so the thread's byte offsets
  // within a block are goff + 4096 j; the block's base is wave-uniform.
  constexpr int RPJ = 256 / CPR;                     // rows per slot index
  const int grow0 = tid / CPR;
  const uint32_t goff = (uint32_t)(grow0 * D + 8 * pf_chunk<D>(grow0, tid % CPR)) * 2u;
  auto dma = [&](int kb) {
    const char* kbase = reinterpret_cast<const char*>(kh + (int64_t)kb * kPfK * D);
    const char* vbase = reinterpret_cast<const char*>(vh + (int64_t)kb * kPfK * D);
    uint16_t* kd = k_s[kb & 1] + 8 * 64 * w;
    uint16_t* vd = v_s[kb & 1] + 8 * 64 * w;
    if ((kb + 1) * kPfK <= a.T) {
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        __builtin_amdgcn_global_load_lds((const void*)(kbase + goff + 4096 * j),
                                         (__attribute__((address_space(3))) void*)(kd + 8 * 256 * j),
                                         16, 0, 0);
        __builtin_amdgcn_global_load_lds((const void*)(vbase + goff + 4096 * j),
                                         (__attribute__((address_space(3))) void*)(vd + 8 * 256 * j),
                                         16, 0, 0);
      }
    } else {                                         // rows past the cache read its last row
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        const int row = RPJ * j + grow0;
        const uint32_t off = goff + 4096u * j -
                             (uint32_t)(row - (min(kb * kPfK + row, a.T - 1) - kb * kPfK)) * (2u * D);
        __builtin_amdgcn_global_load_lds((const void*)(kbase + off),
                                         (__attribute__((address_space(3))) void*)(kd + 8 * 256 * j),
                                         16, 0, 0);
        __builtin_amdgcn_global_load_lds((const void*)(vbase + off),
                                         (__attribute__((address_space(3))) void*)(vd + 8 * 256 * j),
                                         16, 0, 0);
      }
    }
  };

  // One key block.  MASKED: the wavefront's last block (keys past a row, keys
  // past the sequence's end, and the row's own key, which is not gated).  In
  // every earlier block each key precedes every row of the wavefront.  Rows at
  // or past the sequence's end compute on regardless and are cleared when stored.
  auto block = [&](int kb, auto masked_tag) {
    constexpr bool MASKED = decltype(masked_tag)::value;
    const uint16_t* kt = k_s[kb & 1];
    const uint16_t* vt = v_s[kb & 1];

    // S^T: lane holds its queries against keys 16 nb + 4 g4 + i
    f32x4 c[2][4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      c[0][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
      c[1][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kc = 0; kc < KC; ++kc) {
        const int krow = 16 * nb + r16;
        const bf16x8 ka = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(&kt[krow * D + 8 * pf_chunk<D>(krow, 4 * kc + g4)]));
        c[0][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, __builtin_bit_cast(bf16x8, qb[0][kc]),
                                                            c[0][nb], 0, 0, 0);
        c[1][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, __builtin_bit_cast(bf16x8, qb[1][kc]),
                                                            c[1][nb], 0, 0, 0);
      }
    }
    // gate, mask, gated score minus the reference maximum (base-2 units)
    float y[2][16], mx[2];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      mx[hh] = kNegInf;
      const float nm = ADD ? -(C2 + m_i[hh]) : -m_i[hh];
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float cv = c[hh][nb][i];
          const float e = __builtin_amdgcn_exp2f(fmaf(nbs, cv, btau2[hh]));
          const float gs = __builtin_amdgcn_rcpf(fmaf(e, is2, is2));
          float x = ADD ? fmaf(C2is, gs, fmaf(cv, s2, nm)) : fmaf(cv, gs, nm);
          if constexpr (MASKED) {
            const int s = kb * kPfK + 16 * nb + 4 * g4 + i;
            const bool valid = s <= t[hh] && t[hh] < Tb;
            r_i[hh] += valid ? gs : 0.f;
            if (s == t[hh]) x = fmaf(cv, s2, -m_i[hh]);
            x = valid ? x : kNegInf;
          } else {
            r_i[hh] += gs;
          }
          y[hh][4 * nb + i] = x;
          mx[hh] = fmaxf(mx[hh], x);
        }
      mx[hh] = row4_max(mx[hh]);
    }
    // The reference maximum is set by the first block and afterwards moves only
    // when some row's block maximum exceeds it by more than 8 (a wavefront-wide
    // decision): weights stay below 2^8, and the accumulators are rescaled only then.
    if (kb == 0 || __ballot(mx[0] > 8.0f || mx[1] > 8.0f) != 0ull) {
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const float dm = mx[hh] == kNegInf ? 0.f : (kb == 0 ? mx[hh] : fmaxf(mx[hh], 0.f));
        const float alpha = __builtin_amdgcn_exp2f(-dm);
        m_i[hh] += dm;
        l_i[hh] *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) acc[hh][db] *= alpha;
#pragma unroll
        for (int j = 0; j < 16; ++j) y[hh][j] -= dm;
      }
    }
    uint32_t pw[2][8];                     // bf16 pairs: B operands of the two 32-key chunks
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int j = 0; j < 16; j += 2) {
        const float p0 = __builtin_amdgcn_exp2f(y[hh][j]);
        const float p1 = __builtin_amdgcn_exp2f(y[hh][j + 1]);
        l_i[hh] += p0 + p1;
        pw[hh][j / 2] = pack_bf16x2(p0, p1);
      }
    // O^T += V^T P^T over the two 32-key chunks; chunk kk holds keys 4 g4 + j (j < 4)
    // and 16 + 4 g4 + j - 4 (j >= 4), on both operands
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const u32x4 pb0 = {pw[0][4 * kk + 0], pw[0][4 * kk + 1], pw[0][4 * kk + 2], pw[0][4 * kk + 3]};
      const u32x4 pb1 = {pw[1][4 * kk + 0], pw[1][4 * kk + 1], pw[1][4 * kk + 2], pw[1][4 * kk + 3]};
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const int r0 = 32 * kk + vt_row, r1 = r0 + 16;
        const int lc = 2 * db + (vt_c >> 1), half = 4 * (vt_c & 1);
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) i16x4*)(&vt[r0 * D + 8 * pf_chunk<D>(r0, lc) + half]));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) i16x4*)(&vt[r1 * D + 8 * pf_chunk<D>(r1, lc) + half]));
        const u32x4 va = {(uint32_t)(uint16_t)lo[0] | ((uint32_t)(uint16_t)lo[1] << 16),
                          (uint32_t)(uint16_t)lo[2] | ((uint32_t)(uint16_t)lo[3] << 16),
                          (uint32_t)(uint16_t)hi[0] | ((uint32_t)(uint16_t)hi[1] << 16),
                          (uint32_t)(uint16_t)hi[2] | ((uint32_t)(uint16_t)hi[3] << 16)};
        acc[0][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, va),
                                                              __builtin_bit_cast(bf16x8, pb0), acc[0][db], 0, 0, 0);
        acc[1][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, va),
                                                              __builtin_bit_cast(bf16x8, pb1), acc[1][db], 0, 0, 0);
      }
    }
  };

  // Every wavefront passes nkb barriers: this thread's DMA of block kb is done;
  // after the barrier everyone's is, and everyone is done with block kb - 1,
  // whose buffer the next DMA overwrites.
  auto arrive = [&](int kb) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (kb + 1 < nkb) dma(kb + 1);
  };
  if (nkb > 0) dma(0);
  int kb = 0;
  for (; kb + 1 < nkb_w; ++kb) {
    arrive(kb);
    block(kb, std::integral_constant<bool, false>{});
  }
  if (nkb_w > 0) {
    arrive(kb);
    block(kb, std::integral_constant<bool, true>{});
    ++kb;
  }
  for (; kb < nkb; ++kb) arrive(kb);
  // lane holds O[t][16 db + 4 g4 + i]; rows at or past the sequence's end are cleared
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const float ls = row4_sum(l_i[hh]);
    const float rs = row4_sum(r_i[hh]) * is2;
    const int tt = t[hh];
    if (tt < a.T) {
      const bool row_ok = tt < Tb && ls > 0.f;
      const float inv = row_ok ? 1.0f / ls : 0.f;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const uint32_t lo = row_ok ? pack_bf16x2(acc[hh][db][0] * inv, acc[hh][db][1] * inv) : 0u;
        const uint32_t hi = row_ok ? pack_bf16x2(acc[hh][db][2] * inv, acc[hh][db][3] * inv) : 0u;
        *reinterpret_cast<uint2*>(a.out + (qrow0 + tt) * D + 16 * db + 4 * g4) = make_uint2(lo, hi);
      }
      if (g4 == 0) {
        a.R[qrow0 + tt] = tt < Tb ? rs : 0.f;
        a.L[qrow0 + tt] = row_ok ? (m_i[hh] + __log2f(ls)) * 0.6931471805599453f : kNegInf;
      }
    }
  }
}

}  // namespace

hipError_t launch_prefill(const eta_prefill_desc_t& pd, const void* q, const void* k, const void* v,
                          const float* tau, const int32_t* seq_lens, void* out, float* R, float* L,
                          hipStream_t stream, LaunchHook hook) {
  PrefillArgs pa{reinterpret_cast<const uint16_t*>(q), reinterpret_cast<const uint16_t*>(k),
                 reinterpret_cast<const uint16_t*>(v), tau, seq_lens,
                 reinterpret_cast<uint16_t*>(out), R, L, pd.num_q_heads, pd.num_kv_heads,
                 pd.capacity_tokens, pd.beta, pd.C};
  dim3 grid((pd.capacity_tokens + kPfQ - 1) / kPfQ, pd.num_q_heads, pd.batch);
  return with_hook(hook, ETA_KERNEL_PREFILL, stream, [&] {
    if (pd.additive) {
      if (pd.head_dim == 64) hipLaunchKernelGGL((prefill_kernel<64, true>), grid, dim3(256), 0, stream, pa);
      if (pd.head_dim == 128) hipLaunchKernelGGL((prefill_kernel<128, true>), grid, dim3(256), 0, stream, pa);
    } else {
      if (pd.head_dim == 64) hipLaunchKernelGGL((prefill_kernel<64, false>), grid, dim3(256), 0, stream, pa);
      if (pd.head_dim == 128) hipLaunchKernelGGL((prefill_kernel<128, false>), grid, dim3(256), 0, stream, pa);
    }
  });
}

}  // namespace eta
