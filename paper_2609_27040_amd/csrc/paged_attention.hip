// Paged decode attention over the local pool (EMA_LAYOUT_ATTN blocks).
//
// Grid: (split, kv head, sequence). A workgroup of four wavefronts owns one
// 256-token chunk of one sequence for one KV head and computes all G query
// heads that share that KV head (grouped-query attention), so every K/V byte
// is read from HBM once per step.
//   phase 1  scores: 8 lanes per token, 16 channels per lane; packed 16-bit
//            dot products (v_dot2 with fp32 accumulation) and an 8-lane
//            reduction; scores (times scale*log2 e) go to LDS.
//   phase 2  per-head max and exp2 / sum over the chunk (wave reductions).
//   phase 3  P.V: a lane owns channels c and c+64 and reads 8 consecutive
//            tokens of each from the transposed V rows (16 B loads); the
//            probabilities are LDS broadcasts.
//   phase 4  the four waves' partial outputs are summed in LDS; one-chunk
//            sequences write the output, longer ones a split-K partial
//            (unnormalised output, max, sum) merged by a second kernel.
// Tokens at or past the sequence length are masked: their scores are -inf
// and their V elements are zeroed before use, so NaN in unused tail slots
// never reaches the output. Reduction orders depend only on the sequence
// lengths, never on which blocks hold the tokens.
#include "kernels.h"

#include <cmath>

namespace ema {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

constexpr int kD = 128;
constexpr int kCh = kAttnChunk;
constexpr int kWT = kCh / 4;          // tokens per wave

__device__ __forceinline__ u32x4 ld16(const char* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

template <bool BF16>
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  if constexpr (BF16) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a),
                                           __builtin_bit_cast(bf16x2, b), c, false);
  } else {
    return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, a), __builtin_bit_cast(f16x2, b), c,
                                  false);
  }
}

template <bool BF16>
__device__ __forceinline__ float lo16(uint32_t w) {
  if constexpr (BF16) return __builtin_bit_cast(float, w << 16);
  else return float(__builtin_bit_cast(_Float16, uint16_t(w & 0xffffu)));
}
template <bool BF16>
__device__ __forceinline__ float hi16(uint32_t w) {
  if constexpr (BF16) return __builtin_bit_cast(float, w & 0xffff0000u);
  else return float(__builtin_bit_cast(_Float16, uint16_t(w >> 16)));
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ int clamp_len(int len, const AttnArgs& a) {
  const int cap = a.max_blocks * a.block_size;
  return len < 0 ? 0 : (len > cap ? cap : len);
}

template <int G, int BS, bool BF16>
__global__ __launch_bounds__(256) void paged_attn_kernel(AttnArgs a) {
  constexpr int NB = kCh / BS;
  __shared__ int32_t s_ids[NB];
  __shared__ __attribute__((aligned(16))) float s_p[G][kCh];
  __shared__ float s_red[4][G][kD];
  __shared__ float s_m[G], s_l[G];

  const int split = blockIdx.x;
  const int kvh = blockIdx.y;
  const int b = blockIdx.z;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int Hq = a.q_heads;

  const int raw_len = a.seq_lens[b];
  const int len = clamp_len(raw_len, a);
  if (split == 0 && kvh == 0 && threadIdx.x == 0 && len != raw_len && raw_len > 0)
    atomicAdd(a.err_count, 1);
  if (len == 0) {
    if (split == 0)
      for (int e = threadIdx.x; e < G * kD; e += 256)
        a.out[(int64_t(b) * Hq + kvh * G + e / kD) * kD + (e % kD)] = 0.0f;
    return;
  }
  const int n_split_b = (len + kCh - 1) / kCh;
  if (split >= n_split_b) return;
  const int c_start = split * kCh;
  const int nvalid = min(kCh, len - c_start);

  if (threadIdx.x < NB) {
    const int j = c_start / BS + threadIdx.x;
    int id = -1;
    if (j * BS < len) {
      id = a.table[int64_t(b) * a.max_blocks + j];
      if (id < 0 || id >= a.n_local) {
        atomicAdd(a.err_count, 1);
        id = -1;
      }
    }
    s_ids[threadIdx.x] = id;
  }
  __syncthreads();

  const char* pool = a.local;
  const int64_t Bb = a.block_bytes;

  // ---- phase 1: scores -------------------------------------------------------
  {
    const int sub = lane & 7;     // channels sub*16 .. sub*16+15
    const int tok = lane >> 3;    // token within an 8-token pass
    uint32_t qv[G][8];
    const char* qb = reinterpret_cast<const char*>(a.q);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const char* p = qb + ((int64_t(b) * Hq + kvh * G + g) * kD + sub * 16) * 2;
      const u32x4 x = ld16(p), y = ld16(p + 16);
      qv[g][0] = x.x; qv[g][1] = x.y; qv[g][2] = x.z; qv[g][3] = x.w;
      qv[g][4] = y.x; qv[g][5] = y.y; qv[g][6] = y.z; qv[g][7] = y.w;
    }
#pragma unroll
    for (int p0 = 0; p0 < kWT / 8; p0 += 4) {
      u32x4 kx[4], ky[4];
      bool ok[4];
#pragma unroll
      for (int pp = 0; pp < 4; ++pp) {
        const int c = wave * kWT + (p0 + pp) * 8 + tok;
        const int id = s_ids[c / BS];
        ok[pp] = (c < nvalid) && (id >= 0);
        if (ok[pp]) {
          const char* p = pool + int64_t(id) * Bb + (int64_t(kvh * BS + c % BS) * kD + sub * 16) * 2;
          kx[pp] = ld16(p);
          ky[pp] = ld16(p + 16);
        } else {
          kx[pp] = u32x4{0, 0, 0, 0};
          ky[pp] = u32x4{0, 0, 0, 0};
        }
      }
#pragma unroll
      for (int pp = 0; pp < 4; ++pp) {
        const int c = wave * kWT + (p0 + pp) * 8 + tok;
        const uint32_t kk[8] = {kx[pp].x, kx[pp].y, kx[pp].z, kx[pp].w,
                                ky[pp].x, ky[pp].y, ky[pp].z, ky[pp].w};
#pragma unroll
        for (int g = 0; g < G; ++g) {
          float acc = 0.0f;
#pragma unroll
          for (int i = 0; i < 8; ++i) acc = dot2<BF16>(kk[i], qv[g][i], acc);
          acc += __shfl_xor(acc, 1);
          acc += __shfl_xor(acc, 2);
          acc += __shfl_xor(acc, 4);
          if (sub == 0) s_p[g][c] = ok[pp] ? acc * a.scale_log2 : -INFINITY;
        }
      }
    }
  }
  __syncthreads();

  // ---- phase 2: softmax statistics of the chunk ------------------------------
  for (int g = wave; g < G; g += 4) {
    float v[kCh / 64];
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < kCh / 64; ++i) {
      v[i] = s_p[g][lane + 64 * i];
      m = fmaxf(m, v[i]);
    }
    m = wave_max(m);
    float l = 0.0f;
#pragma unroll
    for (int i = 0; i < kCh / 64; ++i) {
      const float p = (m == -INFINITY) ? 0.0f : exp2f(v[i] - m);
      s_p[g][lane + 64 * i] = p;
      l += p;
    }
    l = wave_sum(l);
    if (lane == 0) {
      s_m[g] = m;
      s_l[g] = l;
    }
  }
  __syncthreads();

  // ---- phase 3: P.V ----------------------------------------------------------
  float acc0[G], acc1[G];
#pragma unroll
  for (int g = 0; g < G; ++g) acc0[g] = acc1[g] = 0.0f;
#pragma unroll
  for (int u0 = 0; u0 < kWT / 8; u0 += 4) {
    u32x4 va[4], vb[4];
    int nv[4];
#pragma unroll
    for (int uu = 0; uu < 4; ++uu) {
      const int c0 = wave * kWT + (u0 + uu) * 8;
      const int id = s_ids[c0 / BS];
      const int left = nvalid - c0;
      nv[uu] = id < 0 ? 0 : (left < 0 ? 0 : (left > 8 ? 8 : left));
      if (nv[uu] > 0) {
        const char* p = pool + int64_t(id) * Bb + Bb / 2 +
                        (int64_t(kvh * kD + lane) * BS + c0 % BS) * 2;
        va[uu] = ld16(p);
        vb[uu] = ld16(p + int64_t(64) * BS * 2);
      }
    }
#pragma unroll
    for (int uu = 0; uu < 4; ++uu) {
      if (nv[uu] == 0) continue;
      const int c0 = wave * kWT + (u0 + uu) * 8;
      uint32_t wa[4] = {va[uu].x, va[uu].y, va[uu].z, va[uu].w};
      uint32_t wb[4] = {vb[uu].x, vb[uu].y, vb[uu].z, vb[uu].w};
      if (nv[uu] < 8) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t keep = (2 * q < nv[uu] ? 0xffffu : 0u) |
                                (2 * q + 1 < nv[uu] ? 0xffff0000u : 0u);
          wa[q] &= keep;
          wb[q] &= keep;
        }
      }
      float xa[8], xb[8];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        xa[2 * q] = lo16<BF16>(wa[q]);
        xa[2 * q + 1] = hi16<BF16>(wa[q]);
        xb[2 * q] = lo16<BF16>(wb[q]);
        xb[2 * q + 1] = hi16<BF16>(wb[q]);
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float4 p0 = *reinterpret_cast<const float4*>(&s_p[g][c0]);
        const float4 p1 = *reinterpret_cast<const float4*>(&s_p[g][c0 + 4]);
        const float p[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          acc0[g] = fmaf(p[j], xa[j], acc0[g]);
          acc1[g] = fmaf(p[j], xb[j], acc1[g]);
        }
      }
    }
  }

  // ---- phase 4: merge the four waves and write ------------------------------
#pragma unroll
  for (int g = 0; g < G; ++g) {
    s_red[wave][g][lane] = acc0[g];
    s_red[wave][g][lane + 64] = acc1[g];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < G * kD; e += 256) {
    const int g = e / kD;
    const int c = e % kD;
    const float o = s_red[0][g][c] + s_red[1][g][c] + s_red[2][g][c] + s_red[3][g][c];
    const int hq = kvh * G + g;
    if (n_split_b == 1) {
      a.out[(int64_t(b) * Hq + hq) * kD + c] = s_l[g] > 0.0f ? o / s_l[g] : 0.0f;
    } else {
      const int64_t row = (int64_t(b) * Hq + hq) * a.n_split + split;
      a.part_o[row * kD + c] = o;
      if (c == 0) {
        a.part_ml[row * 2] = s_m[g];
        a.part_ml[row * 2 + 1] = s_l[g];
      }
    }
  }
}

template <int G, int BS>
hipError_t launch_g_bs(const AttnArgs& a, hipStream_t stream) {
  const dim3 grid(a.n_split, a.kv_heads, a.batch);
  if (a.dtype == 1)
    hipLaunchKernelGGL((paged_attn_kernel<G, BS, true>), grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL((paged_attn_kernel<G, BS, false>), grid, dim3(256), 0, stream, a);
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

hipError_t launch_paged_attention(const AttnArgs& a, hipStream_t stream) {
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
