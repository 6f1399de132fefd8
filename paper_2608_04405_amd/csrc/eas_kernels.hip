// Error-Aware Safeguard, prefill side (Sec. 3.2 "Error-Aware Safeguard
// (EAS)", Eq. reconstruction_error): the hard-to-hash set S_err of each
// (sequence, KV head) is the m keys with the largest reconstruction errors
// ||k - h P||, which the prefill kernels already produce (err_out).
//
// One 1024-thread workgroup per (b, h) finds the m-th largest error by a
// three-pass radix select over the 32-bit order key of each float (11, 11
// and 10 bits, most significant first; each pass histograms, in LDS, the keys
// that match the digits fixed so far), then writes, in ascending index
// order, every key above the threshold and the lowest-index keys equal to it
// until m are taken.  The order key maps the IEEE total order of float32 onto
// unsigned integers (negative values complemented, others with the sign bit
// set), so larger errors have larger keys.

#include "bpc_internal.h"

namespace bpc {

constexpr int kHardThreads = 1024;
constexpr int kHardBins = 2048;       // 11-bit digits
constexpr int kHardChunk = 4 * kHardThreads;  // keys per compaction pass

__device__ __forceinline__ uint32_t order_key(uint32_t u) { return (u & 0x80000000u) ? ~u : (u | 0x80000000u); }

__global__ __launch_bounds__(kHardThreads) void select_hard_kernel(const float* __restrict__ err, int64_t sE_b,
                                                                   int64_t sE_h, int Hkv, int N, int m,
                                                                   int32_t* __restrict__ out) {
  __shared__ uint32_t hist[kHardBins];
  __shared__ int wave_tot[kHardThreads / 64];
  __shared__ int found[2];  // digit, keys above it
  const int bh = blockIdx.x;
  const int b = bh / Hkv, h = bh % Hkv;
  const uint32_t* e = reinterpret_cast<const uint32_t*>(err + b * sE_b + h * sE_h);
  const int t = threadIdx.x;

  // ---- the threshold key: `need` = rank of the m-th largest key among the
  // keys that share the digits fixed so far (1 = the largest of them)
  uint32_t prefix = 0u, pmask = 0u;
  int need = m;
  constexpr int kShift[3] = {21, 10, 0}, kBits[3] = {11, 11, 10};
#pragma unroll
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = kShift[pass];
    const uint32_t dmask = (1u << kBits[pass]) - 1u;
    hist[2 * t] = 0u, hist[2 * t + 1] = 0u;
    __syncthreads();
    for (int i = t; i < N; i += kHardThreads) {
      const uint32_t k = order_key(e[i]);
      if ((k & pmask) == prefix) atomicAdd(&hist[(k >> shift) & dmask], 1u);
    }
    __syncthreads();
    // thread t holds bins 2047 - 2t (upper) and 2046 - 2t; the exclusive scan
    // in that order counts the keys in the bins above
    const int hi = (int)hist[kHardBins - 1 - 2 * t], lo = (int)hist[kHardBins - 2 - 2 * t];
    int total;
    const int above_hi = block_exclusive_scan<kHardThreads>(hi + lo, wave_tot, total);
    const int above_lo = above_hi + hi;
    if (above_hi < need && need <= above_hi + hi) found[0] = kHardBins - 1 - 2 * t, found[1] = above_hi;
    if (above_lo < need && need <= above_lo + lo) found[0] = kHardBins - 2 - 2 * t, found[1] = above_lo;
    __syncthreads();
    prefix |= (uint32_t)found[0] << shift;
    pmask |= dmask << shift;
    need -= found[1];
    __syncthreads();  // found[] and hist[] are rewritten by the next pass
  }
  // prefix is the threshold key; `need` keys equal to it are taken, lowest
  // indices first, after the m - need keys above it

  // ---- ordered compaction, kHardChunk keys at a time (four per thread)
  int written = 0, ties_seen = 0;
  for (int c0 = 0; c0 < N; c0 += kHardChunk) {
    uint32_t k[4];
    int nb = 0, nt = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = c0 + 4 * t + u;
      k[u] = (i < N) ? order_key(e[i]) : 0u;
      const bool valid = i < N;
      nb += valid && k[u] > prefix;
      nt += valid && k[u] == prefix;
    }
    int tot;
    const int pre = block_exclusive_scan<kHardThreads>((nt << 16) | nb, wave_tot, tot);
    int tie_rank = ties_seen + (pre >> 16);
    int rank = written + (pre & 0xFFFF) + max(0, min(tie_rank, need) - min(ties_seen, need));
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = c0 + 4 * t + u;
      if (i >= N) break;
      bool keep = k[u] > prefix;
      if (k[u] == prefix) {
        keep = tie_rank < need;
        ++tie_rank;
      }
      if (keep) out[(size_t)bh * m + rank] = i;
      rank += keep;
    }
    written += (tot & 0xFFFF) + max(0, min(ties_seen + (tot >> 16), need) - min(ties_seen, need));
    ties_seen += tot >> 16;
  }
}

hipError_t launch_select_hard(const float* err, int64_t sE_b, int64_t sE_h, int B, int Hkv, int N, int m,
                              int32_t* out, hipStream_t stream) {
  if (m > 0) select_hard_kernel<<<B * Hkv, kHardThreads, 0, stream>>>(err, sE_b, sE_h, Hkv, N, m, out);
  return hipGetLastError();
}

}  // namespace bpc
