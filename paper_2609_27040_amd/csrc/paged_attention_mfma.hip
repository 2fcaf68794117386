// Paged decode attention on the matrix cores (gfx950 MFMA 16x16x32).
//
// With grouped-query attention the G query heads that share a KV head turn
// decode into a small dense contraction per KV head: [G x 128] . [128 x T] for
// the scores and [G x T] . [T x 128] for the output. Both go to
// v_mfma_f32_16x16x32_{bf16,f16} (G <= 16 heads fill one 16-wide tile), which
// leaves the vector ALUs nearly idle and the kernel bound by HBM.
//
// Grid (chunk, KV head, sequence), 4 wavefronts. Each wavefront streams
// 32-token iterations of its share of the chunk with an online softmax:
//   scores   S^T[token][head] = K . Q^T   (A = 16 K rows straight from the
//            block, B = Q^T held in registers; two 16-token tiles whose rows
//            are chosen so that each lane ends up holding 8 consecutive
//            tokens of one head -- exactly the B-operand layout of the next
//            product, so no data moves between lanes)
//   output   O^T[channel][head] += V^T . P^T  (A = 16 channel rows of the
//            transposed V block, 8 consecutive tokens per lane, 16 B loads;
//            P is split into a 16-bit high part and a 16-bit remainder so the
//            probabilities keep ~16 significant bits)
// The four waves' (max, sum, output) are merged in LDS. A sequence longer
// than one chunk writes a partial (unnormalised output, max, sum) that the
// split-K combine kernel merges; merging in-kernel would need device-scope
// fences, which write back and invalidate the whole L2 of an XCD per
// workgroup on this chip. Masked tokens (past the length, or in a block whose id is out of
// range) get -inf scores and zeroed V, so NaN in unused slots never leaks.
// Reduction orders depend only on sequence lengths, not on block ids.
#include "kernels.h"

#include <cmath>

namespace ema {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kD = 128;
constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kIt = 32;                 // tokens per wave iteration
constexpr int kMaxIds = 512 / 16;       // block ids of the largest chunk at the smallest block

__device__ __forceinline__ u32x4 ld16(const char* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

template <bool BF16>
__device__ __forceinline__ f32x4 mfma(u32x4 a, u32x4 b, f32x4 c) {
  if constexpr (BF16)
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// p -> (high, low) 16-bit parts with p ~= high + low.
template <bool BF16>
__device__ __forceinline__ void split16(float p, uint32_t& hi, uint32_t& lo) {
  if constexpr (BF16) {
    const uint32_t u = __builtin_bit_cast(uint32_t, p);
    hi = u >> 16;                                        // truncation: exact remainder
    const float r = p - __builtin_bit_cast(float, u & 0xffff0000u);
    const uint32_t v = __builtin_bit_cast(uint32_t, r);
    lo = (v + 0x7fffu + ((v >> 16) & 1u)) >> 16;         // round to nearest even
  } else {
    const _Float16 h = _Float16(p);
    const _Float16 l = _Float16(p - float(h));
    hi = __builtin_bit_cast(uint16_t, h);
    lo = __builtin_bit_cast(uint16_t, l);
  }
}

__device__ __forceinline__ int clamp_len(int len, const AttnArgs& a) {
  const int cap = a.max_blocks * a.block_size;
  return len < 0 ? 0 : (len > cap ? cap : len);
}

template <int G, int BS, bool BF16>
__global__ __launch_bounds__(kThreads, 3) void attn_mfma_kernel(AttnArgs a) {
  __shared__ int32_t s_ids[kMaxIds];
  __shared__ __attribute__((aligned(16))) float s_o[kWaves][G][kD];
  __shared__ float s_m[kWaves][G], s_l[kWaves][G];

  const int split = blockIdx.x;
  const int kvh = blockIdx.y;
  const int b = blockIdx.z;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int r16 = lane & 15;
  const int q4 = lane >> 4;
  const int Hq = a.q_heads;
  const int chunk = a.chunk;

  const int raw_len = a.seq_lens[b];
  const int len = clamp_len(raw_len, a);
  if (split == 0 && kvh == 0 && tid == 0 && len != raw_len && raw_len > 0)
    atomicAdd(a.err_count, 1);
  if (len == 0) {
    if (split == 0)
      for (int e = tid; e < G * kD; e += kThreads)
        a.out[(int64_t(b) * Hq + kvh * G + e / kD) * kD + (e % kD)] = 0.0f;
    return;
  }
  const int n_split_b = (len + chunk - 1) / chunk;
  if (split >= n_split_b) return;
  const int c_start = split * chunk;
  const int nvalid = min(chunk, len - c_start);
  const int nb = chunk / BS;
  for (int i = tid; i < nb; i += kThreads) {
    const int j = c_start / BS + i;
    int id = -1;
    if (j * BS < len) {
      id = a.table[int64_t(b) * a.max_blocks + j];
      if (id < 0 || id >= a.n_local) {
        atomicAdd(a.err_count, 1);
        id = -1;
      }
    }
    s_ids[i] = id;
  }
  __syncthreads();

  const char* pool = a.local;
  const int64_t Bb = a.block_bytes;

  // Q^T as the B operand: lane (head r16, q4) holds channels 32kk + 8q4 .. +8.
  u32x4 qb[4];
  {
    const char* qrow = reinterpret_cast<const char*>(a.q) +
                       (int64_t(b) * Hq + kvh * G + r16) * kD * 2 + q4 * 16;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      qb[kk] = r16 < G ? ld16(qrow + kk * 64) : u32x4{0, 0, 0, 0};
  }

  float m = -INFINITY;   // running max of this lane's head (log2 domain)
  float lsum = 0.0f;     // this lane's share of the running sum
  f32x4 o[8];
#pragma unroll
  for (int n = 0; n < 8; ++n) o[n] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  const int its = chunk / (kWaves * kIt);
  for (int it = 0; it < its; ++it) {
    const int t0 = (wave * its + it) * kIt;
    if (t0 >= nvalid) break;
    // K rows: tile t, row r16 -> token t0 + 8*(r16/4) + 4t + r16%4.
    u32x4 kr[2][4];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int tok = t0 + 8 * (r16 >> 2) + 4 * t + (r16 & 3);
      const int id = s_ids[tok / BS];
      const bool ok = tok < nvalid && id >= 0;
      const char* p = pool + int64_t(ok ? id : 0) * Bb +
                      (int64_t(kvh * BS + tok % BS) * kD + q4 * 8) * 2;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) kr[t][kk] = ok ? ld16(p + kk * 64) : u32x4{0, 0, 0, 0};
    }
    // V^T rows: d-tile n, row 16n + r16, tokens t0 + 8q4 .. +8 (one block).
    const int vt = t0 + 8 * q4;
    const int vid = s_ids[vt / BS];
    const int vleft = nvalid - vt;
    const int nv = vid < 0 ? 0 : (vleft < 0 ? 0 : (vleft > 8 ? 8 : vleft));
    u32x4 vr[8];
    {
      const char* p = pool + int64_t(nv > 0 ? vid : 0) * Bb + Bb / 2 +
                      (int64_t(kvh * kD + r16) * BS + vt % BS) * 2;
#pragma unroll
      for (int n = 0; n < 8; ++n)
        vr[n] = nv > 0 ? ld16(p + int64_t(16 * n) * BS * 2) : u32x4{0, 0, 0, 0};
      if (nv > 0 && nv < 8) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t keep = (2 * q < nv ? 0xffffu : 0u) | (2 * q + 1 < nv ? 0xffff0000u : 0u);
#pragma unroll
          for (int n = 0; n < 8; ++n) vr[n][q] &= keep;
        }
      }
    }
    // Scores for tokens vt + 4t + i of head r16.
    f32x4 s[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      s[t] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) s[t] = mfma<BF16>(kr[t][kk], qb[kk], s[t]);
    }
    float sv[8];
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      sv[j] = j < nv ? s[j >> 2][j & 3] * a.scale_log2 : -INFINITY;
      mx = fmaxf(mx, sv[j]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m, mx);
    const float alpha = m_new == -INFINITY ? 1.0f : exp2f(m - m_new);
    uint32_t ph[4], pl[4];
    float ps = 0.0f;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float p0 = m_new == -INFINITY ? 0.0f : exp2f(sv[2 * q] - m_new);
      const float p1 = m_new == -INFINITY ? 0.0f : exp2f(sv[2 * q + 1] - m_new);
      ps += p0 + p1;
      uint32_t h0, l0, h1, l1;
      split16<BF16>(p0, h0, l0);
      split16<BF16>(p1, h1, l1);
      ph[q] = h0 | (h1 << 16);
      pl[q] = l0 | (l1 << 16);
    }
    lsum = lsum * alpha + ps;
    m = m_new;
    const u32x4 PH = {ph[0], ph[1], ph[2], ph[3]};
    const u32x4 PL = {pl[0], pl[1], pl[2], pl[3]};
#pragma unroll
    for (int n = 0; n < 8; ++n) {
      o[n] *= alpha;
      o[n] = mfma<BF16>(vr[n], PH, o[n]);
      o[n] = mfma<BF16>(vr[n], PL, o[n]);
    }
  }

  // ---- merge the four waves ------------------------------------------------
  lsum += __shfl_xor(lsum, 16);
  lsum += __shfl_xor(lsum, 32);
  if (r16 < G) {
    if (q4 == 0) {
      s_m[wave][r16] = m;
      s_l[wave][r16] = lsum;
    }
#pragma unroll
    for (int n = 0; n < 8; ++n)
      *reinterpret_cast<f32x4*>(&s_o[wave][r16][16 * n + 4 * q4]) = o[n];
  }
  __syncthreads();
  const bool single = n_split_b == 1;
  for (int e = tid; e < G * kD; e += kThreads) {
    const int g = e / kD;
    const int d = e % kD;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, s_m[w][g]);
    float L = 0.0f, O = 0.0f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float mw = s_m[w][g];
        if (mw == -INFINITY) continue;
        const float f = exp2f(mw - M);
        L = fmaf(f, s_l[w][g], L);
        O = fmaf(f, s_o[w][g][d], O);
      }
    }
    const int hq = kvh * G + g;
    if (single) {
      a.out[(int64_t(b) * Hq + hq) * kD + d] = L > 0.0f ? O / L : 0.0f;
    } else {
      const int64_t row = (int64_t(b) * Hq + hq) * a.n_split + split;
      a.part_o[row * kD + d] = O;
      if (d == 0) {
        a.part_ml[row * 2] = M;
        a.part_ml[row * 2 + 1] = L;
      }
    }
  }
}

template <int G, int BS>
hipError_t launch_g_bs(const AttnArgs& a, hipStream_t stream) {
  const dim3 grid(a.n_split, a.kv_heads, a.batch);
  if (a.dtype == 1)
    hipLaunchKernelGGL((attn_mfma_kernel<G, BS, true>), grid, dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((attn_mfma_kernel<G, BS, false>), grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

template <int G>
hipError_t launch_g(const AttnArgs& a, hipStream_t stream) {
  switch (a.block_size) {
    case 16: return launch_g_bs<G, 16>(a, stream);
    case 32: return launch_g_bs<G, 32>(a, stream);
    case 64: return launch_g_bs<G, 64>(a, stream);
    case 128: return launch_g_bs<G, 128>(a, stream);
    case 256: return launch_g_bs<G, 256>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_paged_attention_mfma(const AttnArgs& a, hipStream_t stream) {
  if (a.batch == 0) return hipSuccess;
  hipError_t e;
  switch (a.q_heads / a.kv_heads) {
    case 1: e = launch_g<1>(a, stream); break;
    case 2: e = launch_g<2>(a, stream); break;
    case 4: e = launch_g<4>(a, stream); break;
    case 8: e = launch_g<8>(a, stream); break;
    case 16: e = launch_g<16>(a, stream); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess || a.n_split <= 1) return e;
  return launch_attn_combine(a, stream);
}

}  // namespace ema
