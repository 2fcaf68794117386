// Split-K merge for paged decode attention.
//
// A sequence longer than one chunk leaves one partial per chunk:
// unnormalised output o_s[128], running max m_s (log2 domain) and sum l_s.
// The result is sum_s 2^(m_s - M) o_s / sum_s 2^(m_s - M) l_s with
// M = max_s m_s. One workgroup of 128 threads per (sequence, query head):
// the split weights are computed once into LDS, then every thread (one
// channel) streams the partial outputs with 16 independent loads in flight,
// so a 64-split merge costs a handful of memory round trips. Summation order
// depends only on the number of splits.
#include "kernels.h"

#include <cmath>

namespace ema {
namespace {

constexpr int kD = 128;
constexpr int kBatch = 16;
constexpr int kLdsSplits = 256;

__device__ __forceinline__ float block_reduce(float v, float* s_buf, bool is_max) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float w = __shfl_xor(v, o);
    v = is_max ? fmaxf(v, w) : v + w;
  }
  if ((threadIdx.x & 63) == 0) s_buf[threadIdx.x >> 6] = v;
  __syncthreads();
  const float r = is_max ? fmaxf(s_buf[0], s_buf[1]) : s_buf[0] + s_buf[1];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kD) void attn_combine_kernel(AttnArgs a) {
  __shared__ float s_w[kLdsSplits];
  __shared__ float s_buf[2];
  const int hq = blockIdx.x;
  const int b = blockIdx.y;
  const int tid = threadIdx.x;
  const int cap = a.max_blocks * a.block_size;
  const int raw = a.seq_lens[b];
  const int len = raw < 0 ? 0 : (raw > cap ? cap : raw);
  const int nsp = (len + a.chunk - 1) / a.chunk;
  if (nsp <= 1) return;
  const int64_t base = (int64_t(b) * a.q_heads + hq) * a.n_split;
  const float* ml = a.part_ml + base * 2;

  float mloc = -INFINITY;
  for (int s = tid; s < nsp; s += kD) mloc = fmaxf(mloc, ml[2 * s]);
  const float M = block_reduce(mloc, s_buf, true);
  float lloc = 0.0f;
  for (int s = tid; s < nsp; s += kD) {
    const float m = ml[2 * s];
    const float w = (M == -INFINITY || m == -INFINITY) ? 0.0f : exp2f(m - M);
    lloc = fmaf(w, ml[2 * s + 1], lloc);
    if (s < kLdsSplits) s_w[s] = w;
  }
  const float L = block_reduce(lloc, s_buf, false);   // its barrier also publishes s_w

  const float* po = a.part_o + base * kD + tid;
  float o = 0.0f;
  for (int s0 = 0; s0 < nsp; s0 += kBatch) {
    float v[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int s = min(s0 + j, nsp - 1);
      v[j] = po[int64_t(s) * kD];
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int s = s0 + j;
      if (s < nsp) {
        float w;
        if (s < kLdsSplits) {
          w = s_w[s];
        } else {
          const float m = ml[2 * s];
          w = (M == -INFINITY || m == -INFINITY) ? 0.0f : exp2f(m - M);
        }
        o = fmaf(w, v[j], o);
      }
    }
  }
  a.out[(int64_t(b) * a.q_heads + hq) * kD + tid] = L > 0.0f ? o / L : 0.0f;
}

}  // namespace

hipError_t launch_attn_combine(const AttnArgs& a, hipStream_t stream) {
  if (a.batch == 0 || a.n_split <= 1) return hipSuccess;
  hipLaunchKernelGGL(attn_combine_kernel, dim3(a.q_heads, a.batch), dim3(kD), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ema
