// Decode-step kernels: query packing, XOR/popcount scoring, exact top-k
// selection and sparse attention over the gathered K/V rows (Sec. 3.2
// "Retrieval Phase"; Algorithm "Computing hashing score"; Appendix "CUDA
// Optimizations on Bitwise Operations"; Sec. 4.2 "Kernel Evaluation").
//
// Selection works on the weighted Hamming distance
//     dist_n = sum_j 2^j popcount(M_j & (code_n XOR s)),   c_n = sum|p| - 2 dist_n,
// so the k largest scores are the k smallest distances, and distances are
// small integers in [0, 127 L].  Pipeline per (sequence b, KV head h):
//   1 qpack      x = sum_g q_g P^T (fp64, fixed order), 7-bit quantisation, 8 bit planes
//   2 scan       per 16384-key slice: distances into LDS, slice histogram, the slice's own
//                k-th smallest distance kth_s, candidates (dist <= kth_s) in key order
//   3 threshold  global k-th smallest distance T* from the slice histograms, the tie quota,
//                and every slice's output offset
//   4 select     every slice writes its selected keys at its offset: ascending key order,
//                ties at T* resolved to the lowest indices
//   5 attend     per 256 selected keys: gather K/V rows, online-softmax partials in fp32
//   6 merge      per query head: log-sum-exp merge of the partials
// The global threshold T* is never above any slice's kth_s (that slice alone already holds
// k keys at or below kth_s), so the candidates contain every selected key, and every
// histogram bin at or below T* was stored by every slice.

#include "bpc_internal.h"

namespace bpc {

// ---------------------------------------------------------------------------
// block-wide exclusive scan of one int per thread (NT threads, wave64)
// ---------------------------------------------------------------------------
template <int NT>
__device__ __forceinline__ int block_exclusive_scan(int v, int* wave_tot, int& total) {
  constexpr int NW = NT / 64;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wave_tot[wid] = x;
  __syncthreads();
  if (wid == 0) {
    int t = (lane < NW) ? wave_tot[lane] : 0;
#pragma unroll
    for (int o = 1; o < NW; o <<= 1) {
      const int y = __shfl_up(t, o, 64);
      if (lane >= o) t += y;
    }
    if (lane < NW) wave_tot[lane] = t;  // inclusive prefix of wave totals
  }
  __syncthreads();
  const int before = (wid > 0) ? wave_tot[wid - 1] : 0;
  total = wave_tot[NW - 1];
  __syncthreads();  // wave_tot may be reused right after
  return before + x - v;
}

// ---------------------------------------------------------------------------
// 1. query projection, quantisation and packing -- one workgroup per (b, h)
// ---------------------------------------------------------------------------
template <int L>
__global__ __launch_bounds__(256) void qpack_kernel(const uint16_t* __restrict__ q, const float* __restrict__ P,
                                                    int64_t sP_b, int64_t sP_h, int Hkv, int G,
                                                    uint32_t* __restrict__ qcode_ws, int* __restrict__ T_ws,
                                                    uint32_t* __restrict__ qcode_out) {
  constexpr int W = L / 32;
  const int bh = blockIdx.x;
  const int b = bh / Hkv, h = bh % Hkv;
  const float* Pb = P + b * sP_b + h * sP_h;
  const uint16_t* qb = q + ((size_t)b * Hkv * G + (size_t)h * G) * kHeadDim;
  __shared__ double xs[kMaxGroup][L];
  __shared__ double xbar[L];
  __shared__ int ps[L];
  __shared__ double mx_s;
  for (int pair = threadIdx.x; pair < G * L; pair += 256) {
    const int g = pair / L, i = pair % L;
    const float* pr = Pb + (size_t)i * kHeadDim;
    const uint16_t* qr = qb + (size_t)g * kHeadDim;
    double blk[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      double acc = 0.0;
      for (int d = 32 * c; d < 32 * c + 32; ++d) acc = dadd(acc, dmul((double)pr[d], bf16_to_f64(qr[d])));
      blk[c] = acc;
    }
    xs[g][i] = dadd(dadd(blk[0], blk[1]), dadd(blk[2], blk[3]));
  }
  __syncthreads();
  if (threadIdx.x < L) {
    double x = xs[0][threadIdx.x];
    for (int g = 1; g < G; ++g) x = dadd(x, xs[g][threadIdx.x]);
    xbar[threadIdx.x] = x;
  }
  __syncthreads();
  if (threadIdx.x < 64) {
    double m = 0.0;
    for (int i = threadIdx.x; i < L; i += 64) m = fmax(m, fabs(xbar[i]));
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) m = fmax(m, __shfl_xor(m, o, 64));
    if (threadIdx.x == 0) mx_s = m;
  }
  __syncthreads();
  const double m = mx_s;
  if (threadIdx.x < L) {
    int p = 0;
    if (m > 0.0) p = (int)round(dmul(xbar[threadIdx.x], 127.0) / m);
    ps[threadIdx.x] = p;
  }
  __syncthreads();
  if (threadIdx.x < 8 * W) {
    const int plane = threadIdx.x / W, word = threadIdx.x % W;
    uint32_t v = 0;
    for (int bit = 0; bit < 32; ++bit) {
      const int p = ps[word * 32 + bit];
      const uint32_t on = (plane == 0) ? (p >= 0 ? 1u : 0u) : ((uint32_t)abs(p) >> (plane - 1)) & 1u;
      v |= on << bit;
    }
    qcode_ws[(size_t)bh * 8 * W + threadIdx.x] = v;
    if (qcode_out) qcode_out[(size_t)bh * 8 * W + threadIdx.x] = v;
  }
  if (threadIdx.x >= 64 && threadIdx.x < 128) {
    int s = 0;
    for (int i = threadIdx.x - 64; i < L; i += 64) s += abs(ps[i]);
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) s += __shfl_xor(s, o, 64);
    if (threadIdx.x == 64) T_ws[bh] = s;
  }
}

// ---------------------------------------------------------------------------
// 2. scan -- one 1024-thread workgroup per 16384-key slice of one (b, h)
// ---------------------------------------------------------------------------
template <int W>
__device__ __forceinline__ void load_code(const uint32_t* p, uint32_t (&c)[W]) {
  if constexpr (W == 1) {
    c[0] = *p;
  } else if constexpr (W == 2) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    c[0] = v.x, c[1] = v.y;
  } else {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    c[0] = v.x, c[1] = v.y, c[2] = v.z, c[3] = v.w;
  }
}

template <int L>
__global__ __launch_bounds__(kScanThreads) void scan_kernel(
    const uint32_t* __restrict__ codes, int64_t sC_b, int64_t sC_h, int Hkv, int N, int k, int nslices,
    const uint32_t* __restrict__ qcode_ws, const int* __restrict__ T_ws, uint32_t* __restrict__ cand,
    int* __restrict__ cand_count, uint16_t* __restrict__ hist_fine, uint32_t* __restrict__ hist_coarse,
    int32_t* __restrict__ score_out) {
  constexpr int W = L / 32;
  constexpr int NB = dist_bins(L);
  constexpr int NBW = (NB + 1) / 2;  // two 16-bit counts per LDS word
  constexpr int PER = kSlice / kScanThreads;
  __shared__ uint16_t dist_s[kSlice];
  __shared__ uint32_t hist_s[NBW];
  __shared__ int wave_tot[kScanThreads / 64];
  __shared__ int kth_s;

  const int s = blockIdx.x, bh = blockIdx.y;
  const int b = bh / Hkv, h = bh % Hkv;
  const int n0 = s * kSlice;
  const int cnt = min(kSlice, N - n0);

  uint32_t sg[W], M[7][W];
  const uint32_t* qc = qcode_ws + (size_t)bh * 8 * W;
#pragma unroll
  for (int w = 0; w < W; ++w) {
    sg[w] = qc[w];
#pragma unroll
    for (int j = 0; j < 7; ++j) M[j][w] = qc[(1 + j) * W + w];
  }
  const int T = T_ws[bh];
  for (int i = threadIdx.x; i < NBW; i += kScanThreads) hist_s[i] = 0;
  if (threadIdx.x == 0) kth_s = NB - 1;
  __syncthreads();

  const uint32_t* cb = codes + b * sC_b + h * sC_h + (int64_t)n0 * W;
  int32_t* so = score_out ? score_out + (size_t)bh * N + n0 : nullptr;
  for (int n = threadIdx.x; n < cnt; n += kScanThreads) {
    uint32_t c[W];
    load_code<W>(cb + (int64_t)n * W, c);
    uint32_t x[W];
#pragma unroll
    for (int w = 0; w < W; ++w) x[w] = c[w] ^ sg[w];
    uint32_t dist = 0;
#pragma unroll
    for (int j = 0; j < 7; ++j) {
      uint32_t pc = 0;
#pragma unroll
      for (int w = 0; w < W; ++w) pc += __popc(M[j][w] & x[w]);
      dist += pc << j;
    }
    dist_s[n] = (uint16_t)dist;
    atomicAdd(&hist_s[dist >> 1], 1u << ((dist & 1u) << 4));
    if (so) so[n] = T - 2 * (int)dist;
  }
  __syncthreads();

  // the slice's k-th smallest distance (all bins if the slice holds < k keys)
  if (cnt >= k) {
    constexpr int BPT = (NB + kScanThreads - 1) / kScanThreads;
    const int t0 = threadIdx.x * BPT;
    int local = 0;
    for (int t = t0; t < min(t0 + BPT, NB); ++t) local += (hist_s[t >> 1] >> ((t & 1) << 4)) & 0xFFFFu;
    int total;
    int before = block_exclusive_scan<kScanThreads>(local, wave_tot, total);
    if (before < k && before + local >= k) {
      int cum = before;
      for (int t = t0; t < min(t0 + BPT, NB); ++t) {
        cum += (hist_s[t >> 1] >> ((t & 1) << 4)) & 0xFFFFu;
        if (cum >= k) {
          kth_s = t;
          break;
        }
      }
    }
    __syncthreads();
  }
  const int kth = kth_s;

  // slice histogram: fine bins [0, kth] (u16) and 128 coarse bins over all of it
  const size_t sl = (size_t)bh * nslices + s;
  uint16_t* hf = hist_fine + sl * fine_stride(L);
  for (int t = threadIdx.x; t <= kth; t += kScanThreads) hf[t] = (uint16_t)((hist_s[t >> 1] >> ((t & 1) << 4)) & 0xFFFFu);
  {
    // 8 threads per coarse bin, 16 fine bins each
    const int cbin = threadIdx.x >> 3, part = threadIdx.x & 7;
    int sum = 0;
    const int t0 = (cbin << kCoarseShift) + part * 16;
    for (int t = t0; t < t0 + 16 && t < NB; ++t) sum += (hist_s[t >> 1] >> ((t & 1) << 4)) & 0xFFFFu;
    sum += __shfl_xor(sum, 1, 64);
    sum += __shfl_xor(sum, 2, 64);
    sum += __shfl_xor(sum, 4, 64);
    if (part == 0) hist_coarse[sl * kCoarseBins + cbin] = (uint32_t)sum;
  }

  // candidates in key order: thread t owns keys [PER t, PER t + PER)
  int mine = 0;
  const int base_n = threadIdx.x * PER;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int n = base_n + e;
    mine += (n < cnt && dist_s[n] <= kth) ? 1 : 0;
  }
  int total;
  int pos = block_exclusive_scan<kScanThreads>(mine, wave_tot, total);
  uint32_t* cs = cand + sl * kSlice;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int n = base_n + e;
    if (n < cnt) {
      const uint32_t d = dist_s[n];
      if ((int)d <= kth) cs[pos++] = ((uint32_t)n << 16) | d;
    }
  }
  if (threadIdx.x == 0) cand_count[sl] = total;
}

// ---------------------------------------------------------------------------
// 3. threshold -- one workgroup per (b, h)
// ---------------------------------------------------------------------------
template <int L>
__global__ __launch_bounds__(256) void threshold_kernel(int k, int nslices, const uint16_t* __restrict__ hist_fine,
                                                        const uint32_t* __restrict__ hist_coarse,
                                                        int* __restrict__ sel_info, int* __restrict__ sel_base,
                                                        int* __restrict__ tie_base) {
  constexpr int NB = dist_bins(L);
  constexpr int FS = fine_stride(L);
  const int bh = blockIdx.x;
  __shared__ int coarse_tot[kCoarseBins];
  __shared__ int fine_tot[1 << kCoarseShift];
  __shared__ int info[4];  // C*, below C*, T*, quota
  const uint32_t* hc = hist_coarse + (size_t)bh * nslices * kCoarseBins;
  const uint16_t* hf = hist_fine + (size_t)bh * nslices * FS;
  if (threadIdx.x < kCoarseBins) {
    int s = 0;
    for (int sl = 0; sl < nslices; ++sl) s += (int)hc[(size_t)sl * kCoarseBins + threadIdx.x];
    coarse_tot[threadIdx.x] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int cum = 0, c = 0;
    for (; c < kCoarseBins - 1; ++c) {
      if (cum + coarse_tot[c] >= k) break;
      cum += coarse_tot[c];
    }
    info[0] = c;
    info[1] = cum;
  }
  __syncthreads();
  const int cstar = info[0];
  if (threadIdx.x < (1 << kCoarseShift)) {
    const int t = (cstar << kCoarseShift) + threadIdx.x;
    int s = 0;
    if (t < NB)
      for (int sl = 0; sl < nslices; ++sl) s += hf[(size_t)sl * FS + t];
    fine_tot[threadIdx.x] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    // bins up to T* are valid in every slice; the scan stops there
    int cum = info[1], t = 0;
    for (; t < (1 << kCoarseShift) - 1; ++t) {
      if (cum + fine_tot[t] >= k) break;
      cum += fine_tot[t];
    }
    const int tstar = min((cstar << kCoarseShift) + t, NB - 1);
    info[2] = tstar;
    info[3] = k - cum;  // ties at T* that are taken
    sel_info[bh * 4 + 0] = tstar;
    sel_info[bh * 4 + 1] = k - cum;
  }
  __syncthreads();
  const int tstar = info[2], quota = info[3];
  // per-slice counts below T* and at T*, then exclusive prefixes over slices
  __shared__ int below_s[256], tie_s[256];
  __shared__ int carry_below, carry_tie;
  if (threadIdx.x == 0) carry_below = 0, carry_tie = 0;
  __syncthreads();
  for (int base = 0; base < nslices; base += 256) {
    const int sl = base + threadIdx.x;
    int below = 0, tie = 0;
    if (sl < nslices) {
      const uint32_t* c = hc + (size_t)sl * kCoarseBins;
      for (int cc = 0; cc < cstar; ++cc) below += (int)c[cc];
      const uint16_t* f = hf + (size_t)sl * FS;
      for (int t = cstar << kCoarseShift; t < tstar; ++t) below += f[t];
      tie = f[tstar];
    }
    below_s[threadIdx.x] = below;
    tie_s[threadIdx.x] = tie;
    __syncthreads();
    if (threadIdx.x == 0) {
      int cb = carry_below, ct = carry_tie;
      for (int i = 0; i < 256 && base + i < nslices; ++i) {
        const int bl = below_s[i], tl = tie_s[i];
        sel_base[(size_t)bh * nslices + base + i] = cb + min(ct, quota);
        tie_base[(size_t)bh * nslices + base + i] = ct;
        cb += bl;
        ct += tl;
      }
      carry_below = cb, carry_tie = ct;
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// 4. select -- one workgroup per slice; writes the slice's selected keys
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void select_kernel(int k, int nslices, const uint32_t* __restrict__ cand,
                                                     const int* __restrict__ cand_count,
                                                     const int* __restrict__ sel_info,
                                                     const int* __restrict__ sel_base,
                                                     const int* __restrict__ tie_base, int32_t* __restrict__ idx) {
  constexpr int PER = 4;
  __shared__ int wave_tot[4];
  const int s = blockIdx.x, bh = blockIdx.y;
  const size_t sl = (size_t)bh * nslices + s;
  const int tstar = sel_info[bh * 4 + 0], quota = sel_info[bh * 4 + 1];
  int out_pos = sel_base[sl];
  int ties_before = tie_base[sl];
  const int cnt = cand_count[sl];
  const uint32_t* cs = cand + sl * kSlice;
  int32_t* ib = idx + (size_t)bh * k;
  const int n0 = s * kSlice;
  for (int base = 0; base < cnt; base += 256 * PER) {
    uint32_t cv[PER];
    int nb = 0, nt = 0;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int i = base + threadIdx.x * PER + e;
      cv[e] = (i < cnt) ? cs[i] : 0xFFFFFFFFu;
      const int d = (int)(cv[e] & 0xFFFFu);
      if (i < cnt) {
        nb += d < tstar;
        nt += d == tstar;
      }
    }
    int tot;
    // one scan of packed (ties << 16 | below): at most 1024 of each per batch
    const int pre = block_exclusive_scan<256>((nt << 16) | nb, wave_tot, tot);
    int below_pre = pre & 0xFFFF, tie_pre = pre >> 16;
    int taken_before = below_pre + max(0, min(ties_before + tie_pre, quota) - min(ties_before, quota));
    int p = out_pos + taken_before;
    int tie_rank = ties_before + tie_pre;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int i = base + threadIdx.x * PER + e;
      if (i < cnt) {
        const int d = (int)(cv[e] & 0xFFFFu);
        bool take = d < tstar;
        if (d == tstar) {
          take = tie_rank < quota;
          ++tie_rank;
        }
        if (take && p < k) ib[p++] = n0 + (int)(cv[e] >> 16);
      }
    }
    const int tb = tot & 0xFFFF, tt = tot >> 16;
    out_pos += tb + max(0, min(ties_before + tt, quota) - min(ties_before, quota));
    ties_before += tt;
  }
}

// ---------------------------------------------------------------------------
// 5. attention over the selected rows -- one workgroup per 256 selected keys
// Sixteen lanes share a key row: lane l16 holds dims [8 l16, 8 l16 + 8) of q,
// K and V, so one 16-byte load per lane fetches four whole rows per wave.
// Logits are kept in base 2 (scaled by sm_scale * log2 e).
// ---------------------------------------------------------------------------
template <int G>
__global__ __launch_bounds__(kAttnThreads) void attend_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
    const uint16_t* __restrict__ V, int64_t sV_b, int64_t sV_h, int64_t sV_n, const int32_t* __restrict__ idx,
    int Hkv, int N, int k, float scale_log2, float* __restrict__ part) {
  constexpr int ROWS_PER_WAVE = kAttnChunk / (kAttnThreads / 64);  // 64
  const int chunk = blockIdx.x, bh = blockIdx.y;
  const int b = bh / Hkv, h = bh % Hkv;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int l16 = lane & 15, rsub = lane >> 4;
  __shared__ float logit_s[G][kAttnChunk];
  __shared__ float red_s[G][4];
  __shared__ float o_s[4][G][kHeadDim];

  float qf[G][8];
  const uint16_t* qb = q + ((size_t)b * Hkv * G + (size_t)h * G) * kHeadDim + 8 * l16;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const uint4 v = *reinterpret_cast<const uint4*>(qb + (size_t)g * kHeadDim);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      qf[g][2 * e] = bf16_to_f32(w[e] & 0xFFFFu);
      qf[g][2 * e + 1] = bf16_to_f32(w[e] >> 16);
    }
  }
  const int j0 = chunk * kAttnChunk;
  const int nrows = min(kAttnChunk, k - j0);
  const int32_t* ib = idx + (size_t)bh * k + j0;
  const uint16_t* Kb = K + b * sK_b + h * sK_h + 8 * l16;
  const uint16_t* Vb = V + b * sV_b + h * sV_h + 8 * l16;

  // pass 1: logits
  for (int it = 0; it < ROWS_PER_WAVE / 4; ++it) {
    const int r = wid * ROWS_PER_WAVE + it * 4 + rsub;
    float acc[G];
#pragma unroll
    for (int g = 0; g < G; ++g) acc[g] = 0.f;
    const int n = (r < nrows) ? ib[r] : -1;
    const bool ok = (unsigned)n < (unsigned)N;  // an index outside the cache is never read
    if (ok) {
      const uint4 v = *reinterpret_cast<const uint4*>(Kb + (int64_t)n * sK_n);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
      float kf[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        kf[2 * e] = bf16_to_f32(w[e] & 0xFFFFu);
        kf[2 * e + 1] = bf16_to_f32(w[e] >> 16);
      }
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[g] = fmaf(qf[g][e], kf[e], acc[g]);
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float a = acc[g];
      a += __shfl_xor(a, 1, 64);
      a += __shfl_xor(a, 2, 64);
      a += __shfl_xor(a, 4, 64);
      a += __shfl_xor(a, 8, 64);
      if (l16 == 0) logit_s[g][r] = ok ? a * scale_log2 : -INFINITY;
    }
  }
  __syncthreads();
  // per-head max and sum over the chunk (each wave reduces its 64 rows)
  float mx[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float m = logit_s[g][wid * 64 + lane];
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    if (lane == 0) red_s[g][wid] = m;
  }
  __syncthreads();
#pragma unroll
  for (int g = 0; g < G; ++g) mx[g] = fmaxf(fmaxf(red_s[g][0], red_s[g][1]), fmaxf(red_s[g][2], red_s[g][3]));
  __syncthreads();
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int r = wid * 64 + lane;
    const float lg = logit_s[g][r];
    float p = (lg == -INFINITY) ? 0.f : exp2f(lg - mx[g]);
    logit_s[g][r] = p;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) p += __shfl_xor(p, o, 64);
    if (lane == 0) red_s[g][wid] = p;
  }
  __syncthreads();

  // pass 2: weighted sum of V rows
  float o[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[g][e] = 0.f;
  for (int it = 0; it < ROWS_PER_WAVE / 4; ++it) {
    const int r = wid * ROWS_PER_WAVE + it * 4 + rsub;
    const int n = (r < nrows) ? ib[r] : -1;
    if ((unsigned)n < (unsigned)N) {
      const uint4 v = *reinterpret_cast<const uint4*>(Vb + (int64_t)n * sV_n);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
      float vf[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        vf[2 * e] = bf16_to_f32(w[e] & 0xFFFFu);
        vf[2 * e + 1] = bf16_to_f32(w[e] >> 16);
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float p = logit_s[g][r];
#pragma unroll
        for (int e = 0; e < 8; ++e) o[g][e] = fmaf(p, vf[e], o[g][e]);
      }
    }
  }
  // reduce the four row groups of the wave, then the four waves
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float x = o[g][e];
      x += __shfl_xor(x, 16, 64);
      x += __shfl_xor(x, 32, 64);
      o[g][e] = x;
    }
  if (rsub == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < 8; ++e) o_s[wid][g][8 * l16 + e] = o[g][e];
  }
  __syncthreads();
  float* pb = part + ((size_t)bh * gridDim.x + chunk) * G * (kHeadDim + 2);
  for (int e = threadIdx.x; e < G * kHeadDim; e += kAttnThreads) {
    const int g = e / kHeadDim, d = e % kHeadDim;
    pb[g * (kHeadDim + 2) + 2 + d] = (o_s[0][g][d] + o_s[1][g][d]) + (o_s[2][g][d] + o_s[3][g][d]);
  }
  if (threadIdx.x < G) {
    const int g = threadIdx.x;
    pb[g * (kHeadDim + 2) + 0] = mx[g];
    pb[g * (kHeadDim + 2) + 1] = (red_s[g][0] + red_s[g][1]) + (red_s[g][2] + red_s[g][3]);
  }
}

// ---------------------------------------------------------------------------
// 6. merge the chunk partials of one query head
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kHeadDim) void merge_kernel(int Hkv, int G, int nchunks, const float* __restrict__ part,
                                                         float* __restrict__ out) {
  const int bq = blockIdx.x;  // b * Hq + query head
  const int Hq = Hkv * G;
  const int b = bq / Hq, jq = bq % Hq;
  const int h = jq / G, g = jq % G;
  const size_t bh = (size_t)b * Hkv + h;
  const float* pb = part + bh * nchunks * G * (kHeadDim + 2) + (size_t)g * (kHeadDim + 2);
  const size_t cstride = (size_t)G * (kHeadDim + 2);
  float M = -INFINITY;
  for (int c = 0; c < nchunks; ++c) M = fmaxf(M, pb[c * cstride]);
  float lsum = 0.f, acc = 0.f;
  for (int c = 0; c < nchunks; ++c) {
    const float w = exp2f(pb[c * cstride] - M);
    lsum = fmaf(pb[c * cstride + 1], w, lsum);
    acc = fmaf(pb[c * cstride + 2 + threadIdx.x], w, acc);
  }
  out[(size_t)bq * kHeadDim + threadIdx.x] = acc / lsum;
}

// ---------------------------------------------------------------------------
template <int L>
static void launch_decode_L(const DecodeArgs& a, const DecodeLayout& lay) {
  const int BH = a.B * a.Hkv;
  uint32_t* qcode = reinterpret_cast<uint32_t*>(a.ws + lay.off_qcode);
  int* T = reinterpret_cast<int*>(a.ws + lay.off_T);
  uint32_t* cand = reinterpret_cast<uint32_t*>(a.ws + lay.off_cand);
  int* cand_count = reinterpret_cast<int*>(a.ws + lay.off_cand_count);
  uint16_t* hist_fine = reinterpret_cast<uint16_t*>(a.ws + lay.off_hist_fine);
  uint32_t* hist_coarse = reinterpret_cast<uint32_t*>(a.ws + lay.off_hist_coarse);
  int* sel_info = reinterpret_cast<int*>(a.ws + lay.off_sel_info);
  int* sel_base = reinterpret_cast<int*>(a.ws + lay.off_sel_base);
  int* tie_base = reinterpret_cast<int*>(a.ws + lay.off_tie_base);
  int32_t* idx = a.idx_out ? a.idx_out : reinterpret_cast<int32_t*>(a.ws + lay.off_idx);
  float* part = reinterpret_cast<float*>(a.ws + lay.off_part);
  hipStream_t st = a.stream;
  auto mark = [&](int i) {
    if (a.events) (void)hipEventRecord(a.events[i], st);
  };

  mark(0);
  qpack_kernel<L><<<BH, 256, 0, st>>>(a.q, a.P, a.sP_b, a.sP_h, a.Hkv, lay.G, qcode, T, a.qcode_out);
  mark(1);
  scan_kernel<L><<<dim3(lay.nslices, BH), kScanThreads, 0, st>>>(a.codes, a.sC_b, a.sC_h, a.Hkv, a.N, a.k,
                                                                lay.nslices, qcode, T, cand, cand_count, hist_fine,
                                                                hist_coarse, a.score_out);
  mark(2);
  threshold_kernel<L><<<BH, 256, 0, st>>>(a.k, lay.nslices, hist_fine, hist_coarse, sel_info, sel_base, tie_base);
  mark(3);
  select_kernel<<<dim3(lay.nslices, BH), 256, 0, st>>>(a.k, lay.nslices, cand, cand_count, sel_info, sel_base,
                                                       tie_base, idx);
  mark(4);
  const float scale_log2 = a.sm_scale * 1.4426950408889634f;
  const dim3 agrid(lay.nchunks, BH);
  switch (lay.G) {
#define BPC_ATTEND_CASE(GG)                                                                                       \
  case GG:                                                                                                        \
    attend_kernel<GG><<<agrid, kAttnThreads, 0, st>>>(a.q, a.K, a.sK_b, a.sK_h, a.sK_n, a.V, a.sV_b, a.sV_h, a.sV_n, \
                                                      idx, a.Hkv, a.N, a.k, scale_log2, part);                        \
    break;
    BPC_ATTEND_CASE(1)
    BPC_ATTEND_CASE(2)
    BPC_ATTEND_CASE(4)
    BPC_ATTEND_CASE(8)
    BPC_ATTEND_CASE(16)
#undef BPC_ATTEND_CASE
    default:
      break;
  }
  mark(5);
  merge_kernel<<<a.B * a.Hq, kHeadDim, 0, st>>>(a.Hkv, lay.G, lay.nchunks, part, a.out);
  mark(6);
}

hipError_t launch_decode(const DecodeArgs& a) {
  const DecodeLayout lay = decode_layout(a.B, a.Hq, a.Hkv, a.N, a.L, a.k);
  switch (a.L) {
    case 32: launch_decode_L<32>(a, lay); break;
    case 64: launch_decode_L<64>(a, lay); break;
    default: launch_decode_L<128>(a, lay); break;
  }
  return hipGetLastError();
}

}  // namespace bpc
