// Split-K merge for paged decode attention.
//
// A sequence longer than one chunk leaves one partial per chunk:
// unnormalised output o_s[128], running max m_s (log2 domain) and sum l_s.
// The result is sum_s 2^(m_s - M) o_s / sum_s 2^(m_s - M) l_s with
// M = max_s m_s. One workgroup of 128 threads per (sequence, query head),
// one thread per channel, merging 16 splits per memory round trip with an
// online rescale; no barriers. Summation order depends only on the number of
// splits.
#include "attn_store.h"
#include "kernels.h"

#include <cmath>

namespace ema {
namespace {

constexpr int kD = 128;
constexpr int kBatch = 16;

__global__ __launch_bounds__(kD) void attn_combine_kernel(AttnArgs a) {
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
  const float* po = a.part_o + base * kD + tid;
  // Every thread (one channel) merges all splits online, kBatch at a time:
  // the (max, sum) pairs and its channel of each partial are loaded together.
  float M = -INFINITY, L = 0.0f, O = 0.0f;
  for (int s0 = 0; s0 < nsp; s0 += kBatch) {
    float mm[kBatch], ll[kBatch], oo[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int s = min(s0 + j, nsp - 1);
      mm[j] = ml[2 * s];
      ll[j] = ml[2 * s + 1];
      oo[j] = po[int64_t(s) * kD];
    }
    float Mb = M;
#pragma unroll
    for (int j = 0; j < kBatch; ++j)
      if (s0 + j < nsp) Mb = fmaxf(Mb, mm[j]);
    if (Mb == -INFINITY) continue;
    const float f_old = M == -INFINITY ? 0.0f : exp2f(M - Mb);
    L *= f_old;
    O *= f_old;
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      if (s0 + j >= nsp || mm[j] == -INFINITY) continue;
      const float f = exp2f(mm[j] - Mb);
      L = fmaf(f, ll[j], L);
      O = fmaf(f, oo[j], O);
    }
    M = Mb;
  }
  store_out(a, (int64_t(b) * a.q_heads + hq) * kD + tid, L > 0.0f ? O / L : 0.0f);
}

}  // namespace

hipError_t launch_attn_combine(const AttnArgs& a, hipStream_t stream) {
  if (a.batch == 0 || a.n_split <= 1) return hipSuccess;
  hipLaunchKernelGGL(attn_combine_kernel, dim3(a.q_heads, a.batch), dim3(kD), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ema
