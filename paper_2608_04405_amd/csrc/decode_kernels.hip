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
//                k-th smallest distance kth_s, prefix-form histograms up to kth_s, and the
//                candidates (dist <= kth_s) in key order
//   3 threshold  global k-th smallest distance T*, the tie quota, and each slice's offsets
//   4 select     per slice: its selected keys, written at the slice's offset (ascending key
//                order; ties at T* go to the lowest indices)
//   5 attend     per 128 selected keys: gather the K/V rows, softmax partials in fp32
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

// lowest set lane of a 64-bit ballot, or 64
__device__ __forceinline__ int first_lane(unsigned long long m) { return m ? __ffsll((long long)m) - 1 : 64; }

// ---------------------------------------------------------------------------
// 1. query projection, quantisation and packing -- one workgroup per (b, h)
// P and q are staged in LDS; each fixed-order dot is split over a quad of
// lanes (lane c sums coordinates [32c, 32c + 32) in ascending order) and the
// quad combines its block sums as ((b0 + b1) + (b2 + b3)).
// ---------------------------------------------------------------------------
template <int L>
__global__ __launch_bounds__(256) void qpack_kernel(const uint16_t* __restrict__ q, const float* __restrict__ P,
                                                    int64_t sP_b, int64_t sP_h, int Hkv, int G,
                                                    uint32_t* __restrict__ qcode_ws, int* __restrict__ T_ws,
                                                    uint32_t* __restrict__ qcode_out) {
  constexpr int W = L / 32;
  constexpr int PADB = 33;  // 32 coordinates per block + 1 to skew LDS banks
  const int bh = blockIdx.x;
  const int b = bh / Hkv, h = bh % Hkv;
  const float* Pb = P + b * sP_b + h * sP_h;
  const uint16_t* qb = q + ((size_t)b * Hkv * G + (size_t)h * G) * kHeadDim;
  __shared__ float P_s[L][4][PADB];
  __shared__ float q_s[kMaxGroup][4][PADB];
  __shared__ double x_s[kMaxGroup][L];
  __shared__ double xbar_s[L];
  __shared__ double mx_s;
  __shared__ int tsum_s[2];
  {
    // every global load is issued before the first LDS store
    constexpr int PV = L * kHeadDim / 4 / 256;  // float4 per thread
    float4 pv[PV];
#pragma unroll
    for (int r = 0; r < PV; ++r) pv[r] = reinterpret_cast<const float4*>(Pb)[r * 256 + threadIdx.x];
    const bool has_q = threadIdx.x < G * kHeadDim / 8;
    const uint4 qv = has_q ? reinterpret_cast<const uint4*>(qb)[threadIdx.x] : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int r = 0; r < PV; ++r) {
      const int e = 4 * (r * 256 + threadIdx.x);
      const int i = e >> 7, d = e & 127;
      float* dst = &P_s[i][d >> 5][d & 31];
      dst[0] = pv[r].x, dst[1] = pv[r].y, dst[2] = pv[r].z, dst[3] = pv[r].w;
    }
    if (has_q) {
      const int e = 8 * threadIdx.x;
      const int g = e >> 7, d = e & 127;
      float* dst = &q_s[g][d >> 5][d & 31];
      const uint32_t w[4] = {qv.x, qv.y, qv.z, qv.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        dst[2 * j] = bf16_to_f32(w[j] & 0xFFFFu);
        dst[2 * j + 1] = bf16_to_f32(w[j] >> 16);
      }
    }
  }
  __syncthreads();
  const int ntriples = G * L * 4;
  for (int base = 0; base < ntriples; base += 256) {
    const int tr = base + threadIdx.x;
    const bool valid = tr < ntriples;
    const int c = tr & 3, gi = valid ? (tr >> 2) : 0;
    const int g = gi / L, i = gi % L;
    double acc = 0.0;
#pragma unroll 8
    for (int e = 0; e < 32; ++e) acc = dadd(acc, dmul((double)P_s[i][c][e], (double)q_s[g][c][e]));
    const double s01 = dadd(acc, __shfl_xor(acc, 1, 64));
    const double a = dadd(s01, __shfl_xor(s01, 2, 64));
    if (valid && c == 0) x_s[g][i] = a;
  }
  __syncthreads();
  if (threadIdx.x < L) {
    double x = x_s[0][threadIdx.x];
    for (int g = 1; g < G; ++g) x = dadd(x, x_s[g][threadIdx.x]);
    xbar_s[threadIdx.x] = x;
  }
  __syncthreads();
  if (threadIdx.x < 64) {
    double m = 0.0;
    for (int i = threadIdx.x; i < L; i += 64) m = fmax(m, fabs(xbar_s[i]));
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) m = fmax(m, __shfl_xor(m, o, 64));
    if (threadIdx.x == 0) mx_s = m;
  }
  __syncthreads();
  const double m = mx_s;
  if (threadIdx.x < 128) {  // waves 0 and 1 cover i < L <= 128
    const int i = threadIdx.x;
    int p = 0;
    if (i < L && m > 0.0) p = (int)round(dmul(xbar_s[i], 127.0) / m);
    const uint32_t mag = (uint32_t)abs(p);
    const int wid = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
    for (int plane = 0; plane < 8; ++plane) {
      const bool on = (i < L) && (plane == 0 ? (p >= 0) : (((mag >> (plane - 1)) & 1u) != 0u));
      const unsigned long long mask = __ballot(on);
      if (lane < 2 && 2 * wid + lane < W) {
        const uint32_t word = (uint32_t)(mask >> (32 * lane));
        qcode_ws[(size_t)bh * 8 * W + plane * W + 2 * wid + lane] = word;
        if (qcode_out) qcode_out[(size_t)bh * 8 * W + plane * W + 2 * wid + lane] = word;
      }
    }
    int s = (int)mag;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) s += __shfl_xor(s, o, 64);
    if (lane == 0) tsum_s[wid] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) T_ws[bh] = tsum_s[0] + tsum_s[1];
}

// ---------------------------------------------------------------------------
// 2. scan -- one 1024-thread workgroup per 16384-key slice of one (b, h)
// ---------------------------------------------------------------------------
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// codes are streamed once per step: non-temporal loads keep them from
// displacing reusable lines in the caches
template <int W>
__device__ __forceinline__ void load_code(const uint32_t* p, uint32_t (&c)[W]) {
  if constexpr (W == 1) {
    c[0] = __builtin_nontemporal_load(p);
  } else if constexpr (W == 2) {
    const u32x2_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p));
    c[0] = v.x, c[1] = v.y;
  } else {
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    c[0] = v.x, c[1] = v.y, c[2] = v.z, c[3] = v.w;
  }
}

template <int L>
__global__ __launch_bounds__(kScanThreads) void scan_kernel(
    const uint32_t* __restrict__ codes, int64_t sC_b, int64_t sC_h, int Hkv, int N, int k, int nslices,
    const uint32_t* __restrict__ qcode_ws, const int* __restrict__ T_ws, uint32_t* __restrict__ cand,
    int* __restrict__ cand_count, uint32_t* __restrict__ hist_fine, uint32_t* __restrict__ hist_cc,
    int32_t* __restrict__ score_out) {
  constexpr int W = L / 32;
  constexpr int NB = dist_bins(L);
  constexpr int NBW = (NB + 1) / 2;  // two 16-bit counts per LDS word
  constexpr int PER = kSlice / kScanThreads;
  __shared__ uint16_t dist_s[kSlice];
  __shared__ uint32_t hist_s[NBW];
  __shared__ uint32_t coarse_s[kCoarseBins];
  __shared__ uint32_t cc_s[kCoarseBins + 1];
  __shared__ int wave_tot[kScanThreads / 64];
  __shared__ int cs_s, kth_sh;

  const int s = blockIdx.x, bh = blockIdx.y;
  const int b = bh / Hkv, h = bh % Hkv;
  const int n0 = s * kSlice;
  const int cnt = min(kSlice, N - n0);
  const int lane = threadIdx.x & 63;

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
  __syncthreads();

  // every code load of this thread is issued before the first is consumed;
  // thread t owns keys {K0 + it * KSTEP + t * KPL + u}: KPL keys per 16-byte load
  constexpr int KPL = (W == 4) ? 1 : (W == 2 ? 2 : 4);
  constexpr int NLD = PER / KPL;
  constexpr int KSTEP = kScanThreads * KPL;
  const uint32_t* cb = codes + b * sC_b + h * sC_h + (int64_t)n0 * W;
  u32x4_t cw[NLD];
  const bool full = (cnt == kSlice);
  // a head's codes are W-word aligned; 16-byte loads need a 16-byte aligned base
  const bool vec_ok = (reinterpret_cast<uintptr_t>(cb) & 15u) == 0;
#pragma unroll
  for (int it = 0; it < NLD; ++it) {
    const int n = it * KSTEP + threadIdx.x * KPL;
    if (vec_ok && (full || n + KPL <= cnt)) {
      cw[it] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(cb + (int64_t)n * W));
    } else {
      uint32_t t4[4] = {0u, 0u, 0u, 0u};
      for (int u = 0; u < KPL; ++u)
        if (n + u < cnt)
          for (int w = 0; w < W; ++w) t4[u * W + w] = cb[(int64_t)(n + u) * W + w];
      cw[it] = u32x4_t{t4[0], t4[1], t4[2], t4[3]};
    }
  }
#pragma unroll
  for (int it = 0; it < NLD; ++it) {
#pragma unroll
    for (int u = 0; u < KPL; ++u) {
      const int n = it * KSTEP + threadIdx.x * KPL + u;
      uint32_t dist = 0;
#pragma unroll
      for (int j = 0; j < 7; ++j) {
        uint32_t pc = 0;
#pragma unroll
        for (int w = 0; w < W; ++w) pc += __popc(M[j][w] & (cw[it][u * W + w] ^ sg[w]));
        dist += pc << j;
      }
      if (full || n < cnt) {
        dist_s[n] = (uint16_t)dist;
        atomicAdd(&hist_s[dist >> 1], 1u << ((dist & 1u) << 4));
      }
    }
  }
  __syncthreads();
  if (score_out) {  // debug output, from LDS
    int32_t* so = score_out + (size_t)bh * N + n0;
    for (int n = threadIdx.x; n < cnt; n += kScanThreads) so[n] = T - 2 * (int)dist_s[n];
  }

  // eight threads per coarse bin, sixteen fine bins each: counts and the
  // prefix within the coarse bin
  const int cbin = threadIdx.x >> 3, part = threadIdx.x & 7;
  const int fb0 = (cbin << kCoarseShift) + part * 16;
  uint32_t cntv[16];
  int local = 0;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int t = fb0 + e;
    cntv[e] = (t < NB) ? ((hist_s[t >> 1] >> ((t & 1) << 4)) & 0xFFFFu) : 0u;
    local += (int)cntv[e];
  }
  int incl = local;
#pragma unroll
  for (int o = 1; o < 8; o <<= 1) {
    const int y = __shfl_up(incl, o, 64);
    if (part >= o) incl += y;
  }
  const int pre = incl - local;
  if (part == 7) coarse_s[cbin] = (uint32_t)incl;
  __syncthreads();

  // wave 0: coarse prefix, and the coarse bin holding the slice's k-th key
  if (threadIdx.x < 64) {
    const uint32_t c0 = coarse_s[2 * lane], c1 = coarse_s[2 * lane + 1];
    int x = (int)(c0 + c1);
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    const int ex = x - (int)(c0 + c1);
    cc_s[2 * lane] = (uint32_t)ex;
    cc_s[2 * lane + 1] = (uint32_t)ex + c0;
    if (lane == 63) cc_s[kCoarseBins] = (uint32_t)x;
    const unsigned long long m0 = __ballot(ex + (int)c0 >= k);
    const unsigned long long m1 = __ballot(x >= k);
    const int f0 = first_lane(m0), f1 = first_lane(m1);
    // lowest coarse bin whose inclusive prefix reaches k
    const int cs = min(f0 < 64 ? 2 * f0 : 1 << 30, f1 < 64 ? 2 * f1 + 1 : 1 << 30);
    if (lane == 0) {
      cs_s = (cnt >= k) ? cs : -1;
      kth_sh = NB - 1;
    }
  }
  __syncthreads();
  const int cs = cs_s;
  if (cs >= 0 && cbin == cs) {
    // the eight owners of that coarse bin find the fine bin where the count reaches k
    int cum = (int)cc_s[cs] + pre;
    int found = 1 << 30;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      cum += (int)cntv[e];
      if (cum >= k && found == (1 << 30)) found = fb0 + e;
    }
    if (found != (1 << 30)) atomicMin(&kth_sh, found);
  }
  __syncthreads();
  const int kth = kth_sh;

  // prefix-form histograms: coarse prefix (129 entries) and fine bins <= kth
  const size_t sl = (size_t)bh * nslices + s;
  if (threadIdx.x <= kCoarseBins) hist_cc[sl * kCoarseStride + threadIdx.x] = cc_s[threadIdx.x];
  {
    uint32_t* hf = hist_fine + sl * fine_stride(L);
    uint32_t run = (uint32_t)pre;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int t = fb0 + e;
      if (t <= kth) hf[t] = (run << 16) | cntv[e];
      run += cntv[e];
    }
  }

  // candidates in key order: thread t owns keys [PER t, PER t + PER), read
  // from LDS as two 16-byte vectors
  static_assert(PER == 16, "the candidate pass reads 16 distances per thread");
  uint32_t dw[8];
  {
    const uint4* dv = reinterpret_cast<const uint4*>(dist_s) + 2 * threadIdx.x;
    const uint4 a = dv[0], c = dv[1];
    dw[0] = a.x, dw[1] = a.y, dw[2] = a.z, dw[3] = a.w, dw[4] = c.x, dw[5] = c.y, dw[6] = c.z, dw[7] = c.w;
  }
  const int base_n = threadIdx.x * PER;
  int mine = 0;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int d = (int)((dw[e >> 1] >> ((e & 1) << 4)) & 0xFFFFu);
    mine += (base_n + e < cnt && d <= kth) ? 1 : 0;
  }
  int total;
  int pos = block_exclusive_scan<kScanThreads>(mine, wave_tot, total);
  uint32_t* cs_out = cand + sl * kSlice;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const uint32_t d = (dw[e >> 1] >> ((e & 1) << 4)) & 0xFFFFu;
    if (base_n + e < cnt && (int)d <= kth) cs_out[pos++] = ((uint32_t)(base_n + e) << 16) | d;
  }
  if (threadIdx.x == 0) cand_count[sl] = total;
}

// ---------------------------------------------------------------------------
// 3. threshold -- one workgroup per (b, h)
// ---------------------------------------------------------------------------
template <int L>
__global__ __launch_bounds__(256) void threshold_kernel(int k, int nslices, const uint32_t* __restrict__ hist_fine,
                                                        const uint32_t* __restrict__ hist_cc,
                                                        int* __restrict__ sel_info, int* __restrict__ sel_base,
                                                        int* __restrict__ tie_base) {
  constexpr int NB = dist_bins(L);
  constexpr int FS = fine_stride(L);
  const int bh = blockIdx.x;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  __shared__ int gp_s[kCoarseBins];
  __shared__ int fe_s[1 << kCoarseShift];
  __shared__ int first_s[2];
  __shared__ int wave_tot[4];
  __shared__ int carry_s[2];
  const uint32_t* ccb = hist_cc + (size_t)bh * nslices * kCoarseStride;
  const uint32_t* hfb = hist_fine + (size_t)bh * nslices * FS;

  // coarse: GP(c + 1) = keys of all slices with distance < 128 (c + 1)
  if (threadIdx.x < kCoarseBins) {
    int acc = 0;
#pragma unroll 4
    for (int sl = 0; sl < nslices; ++sl) acc += (int)ccb[(size_t)sl * kCoarseStride + threadIdx.x + 1];
    gp_s[threadIdx.x] = acc;
    const unsigned long long m = __ballot(acc >= k);
    if (lane == 0) first_s[wid] = m ? first_lane(m) + 64 * wid : (1 << 30);
  }
  __syncthreads();
  const int cstar = min(min(first_s[0], first_s[1]), kCoarseBins - 1);
  const int below_c = (cstar > 0) ? gp_s[cstar - 1] : 0;
  __syncthreads();
  // fine bins of coarse bin C*: inclusive prefix within the bin, summed over slices
  if (threadIdx.x < (1 << kCoarseShift)) {
    const int t = (cstar << kCoarseShift) + threadIdx.x;
    int inc = 0, exc = 0;
    if (t < NB) {
#pragma unroll 4
      for (int sl = 0; sl < nslices; ++sl) {
        const uint32_t v = hfb[(size_t)sl * FS + t];
        exc += (int)(v >> 16);
        inc += (int)(v >> 16) + (int)(v & 0xFFFFu);
      }
    }
    fe_s[threadIdx.x] = exc;
    const unsigned long long m = __ballot(t < NB && below_c + inc >= k);
    if (lane == 0) first_s[wid] = m ? first_lane(m) + 64 * wid : (1 << 30);
  }
  __syncthreads();
  const int tt = min(min(first_s[0], first_s[1]), (1 << kCoarseShift) - 1);
  const int tstar = min((cstar << kCoarseShift) + tt, NB - 1);
  const int below = below_c + fe_s[tt];
  const int quota = k - below;
  if (threadIdx.x == 0) {
    sel_info[bh * 4 + 0] = tstar;
    sel_info[bh * 4 + 1] = quota;
    carry_s[0] = carry_s[1] = 0;
  }
  __syncthreads();
  // per slice: keys below T* and ties at T*; exclusive prefixes over slices
  for (int base = 0; base < nslices; base += 256) {
    const int sl = base + threadIdx.x;
    int bl = 0, ti = 0;
    if (sl < nslices) {
      const uint32_t v = hfb[(size_t)sl * FS + tstar];
      bl = (int)ccb[(size_t)sl * kCoarseStride + cstar] + (int)(v >> 16);
      ti = (int)(v & 0xFFFFu);
    }
    int tb, tt2;
    const int pb = block_exclusive_scan<256>(bl, wave_tot, tb);
    const int pt = block_exclusive_scan<256>(ti, wave_tot, tt2);
    const int cb = carry_s[0], ct = carry_s[1];
    if (sl < nslices) {
      sel_base[(size_t)bh * nslices + sl] = cb + pb + min(ct + pt, quota);
      tie_base[(size_t)bh * nslices + sl] = ct + pt;
    }
    __syncthreads();
    if (threadIdx.x == 0) carry_s[0] = cb + tb, carry_s[1] = ct + tt2;
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// 4. select -- one workgroup per slice; writes the slice's selected keys at
// its offset, in ascending key order
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kSelectThreads) void select_kernel(int k, int nslices, const uint32_t* __restrict__ cand,
                                                               const int* __restrict__ cand_count,
                                                               const int* __restrict__ sel_info,
                                                               const int* __restrict__ sel_base,
                                                               const int* __restrict__ tie_base,
                                                               int32_t* __restrict__ idx) {
  constexpr int PER = 16;
  __shared__ int wave_tot[kSelectThreads / 64];
  const int s = blockIdx.x, bh = blockIdx.y;
  const size_t sl = (size_t)bh * nslices + s;
  const int tstar = sel_info[bh * 4 + 0], quota = sel_info[bh * 4 + 1];
  int out_pos = sel_base[sl];
  int ties_before = tie_base[sl];
  const int cnt = cand_count[sl];
  const uint32_t* cs = cand + sl * kSlice;
  int32_t* ib = idx + (size_t)bh * k;
  const int n0 = s * kSlice;
  for (int base = 0; base < cnt; base += kSelectThreads * PER) {
    const int i0 = base + threadIdx.x * PER;
    uint32_t cv[PER];
    if (i0 + PER <= cnt) {
      const uint4* v = reinterpret_cast<const uint4*>(cs + i0);
#pragma unroll
      for (int r = 0; r < PER / 4; ++r) {
        const uint4 x = v[r];
        cv[4 * r] = x.x, cv[4 * r + 1] = x.y, cv[4 * r + 2] = x.z, cv[4 * r + 3] = x.w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < PER; ++e) cv[e] = (i0 + e < cnt) ? cs[i0 + e] : 0xFFFFFFFFu;
    }
    int nb = 0, nt = 0;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int d = (int)(cv[e] & 0xFFFFu);  // padding entries carry 0xFFFF, above any T*
      nb += d < tstar;
      nt += d == tstar;
    }
    int tot;
    // one scan of packed (ties << 16 | below): at most 4096 of each per batch
    const int pre = block_exclusive_scan<kSelectThreads>((nt << 16) | nb, wave_tot, tot);
    const int below_pre = pre & 0xFFFF, tie_pre = pre >> 16;
    int p = out_pos + below_pre + max(0, min(ties_before + tie_pre, quota) - min(ties_before, quota));
    int tie_rank = ties_before + tie_pre;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int d = (int)(cv[e] & 0xFFFFu);
      bool take = d < tstar;
      if (d == tstar) {
        take = tie_rank < quota;
        ++tie_rank;
      }
      if (take && p < k) ib[p++] = n0 + (int)(cv[e] >> 16);
    }
    const int tb = tot & 0xFFFF, tt = tot >> 16;
    out_pos += tb + max(0, min(ties_before + tt, quota) - min(ties_before, quota));
    ties_before += tt;
  }
}

// ---------------------------------------------------------------------------
// 5. attention over the selected rows -- one workgroup per 128 selected keys
// Sixteen lanes share a key row (lane l16 holds dims [8 l16, 8 l16 + 8)),
// four rows per wavefront instruction, 32 rows per wavefront; the wavefront
// loads its 32 row indices once and issues every K and V row load before
// the first is consumed.  Logits are kept in base 2 (sm_scale * log2 e).
// The last workgroup of a (b, h) to finish merges the chunk partials.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// a + (bf16 pair x) . (bf16 pair y), fp32 accumulation
__device__ __forceinline__ float dot2_bf16(uint32_t x, uint32_t y, float a) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, x), __builtin_bit_cast(bf16x2_t, y), a, false);
}

// sum over each row of 16 lanes, every lane of the row receives it (DPP)
__device__ __forceinline__ float row16_sum(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x141, 0xF, 0xF, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x140, 0xF, 0xF, false));
  return v;
}

__device__ __forceinline__ void unpack8(const uint4 v, float (&f)[8]) {
  f[0] = bf16_to_f32(v.x & 0xFFFFu), f[1] = bf16_to_f32(v.x >> 16);
  f[2] = bf16_to_f32(v.y & 0xFFFFu), f[3] = bf16_to_f32(v.y >> 16);
  f[4] = bf16_to_f32(v.z & 0xFFFFu), f[5] = bf16_to_f32(v.z >> 16);
  f[6] = bf16_to_f32(v.w & 0xFFFFu), f[7] = bf16_to_f32(v.w >> 16);
}

template <int G>
__global__ __launch_bounds__(kAttnThreads) void attend_kernel(
    int N, int k, int Hkv, int nchunks, const int32_t* __restrict__ idx, const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ K, int64_t sK_b, int64_t sK_h, int64_t sK_n, const uint16_t* __restrict__ V,
    int64_t sV_b, int64_t sV_h, int64_t sV_n, float scale_log2, float* __restrict__ part) {
  constexpr int RPW = kAttnChunk / (kAttnThreads / 64);  // rows per wavefront (32)
  constexpr int SLOTS = RPW / 4;                          // rows per lane (8)
  const int chunk = blockIdx.x, bh = blockIdx.y;
  const int b = bh / Hkv, h = bh % Hkv;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int l16 = lane & 15, rsub = lane >> 4;
  __shared__ float lg_s[G][kAttnChunk];
  __shared__ float red_s[G][4];
  __shared__ float sum_s[G][4];
  __shared__ float o_s[4][G][kHeadDim];

  const int j0 = chunk * kAttnChunk + wid * RPW;  // first selected row of this wavefront
  const int nrows = max(0, min(RPW, k - j0));
  const int myidx = (lane < nrows) ? idx[(size_t)bh * k + j0 + lane] : -1;
  const uint16_t* Kb = K + b * sK_b + h * sK_h + 8 * l16;
  const uint16_t* Vb = V + b * sV_b + h * sV_h + 8 * l16;
  int rown[SLOTS];
#pragma unroll
  for (int it = 0; it < SLOTS; ++it) rown[it] = __shfl(myidx, it * 4 + rsub, 64);
  uint4 kv[SLOTS], vv[SLOTS];
#pragma unroll
  for (int it = 0; it < SLOTS; ++it)
    kv[it] = ((unsigned)rown[it] < (unsigned)N) ? *reinterpret_cast<const uint4*>(Kb + (int64_t)rown[it] * sK_n)
                                               : make_uint4(0, 0, 0, 0);
  if constexpr (G <= 4) {
#pragma unroll
    for (int it = 0; it < SLOTS; ++it)
      vv[it] = ((unsigned)rown[it] < (unsigned)N) ? *reinterpret_cast<const uint4*>(Vb + (int64_t)rown[it] * sV_n)
                                                 : make_uint4(0, 0, 0, 0);
  }
  uint4 qp[G];  // eight bf16 of each query head, as four packed pairs
  {
    const uint16_t* qb = q + ((size_t)b * Hkv * G + (size_t)h * G) * kHeadDim + 8 * l16;
#pragma unroll
    for (int g = 0; g < G; ++g) qp[g] = *reinterpret_cast<const uint4*>(qb + (size_t)g * kHeadDim);
  }

  // logits: packed bf16 dot products (exact products, fp32 sums), then a
  // DPP sum over the 16 lanes of the row
#pragma unroll
  for (int it = 0; it < SLOTS; ++it) {
    const int r = it * 4 + rsub;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float a = dot2_bf16(kv[it].x, qp[g].x, 0.f);
      a = dot2_bf16(kv[it].y, qp[g].y, a);
      a = dot2_bf16(kv[it].z, qp[g].z, a);
      a = dot2_bf16(kv[it].w, qp[g].w, a);
      a = row16_sum(a);
      if (l16 == 0) lg_s[g][wid * RPW + r] = ((unsigned)rown[it] < (unsigned)N) ? a * scale_log2 : -INFINITY;
    }
  }
  if constexpr (G > 4) {
#pragma unroll
    for (int it = 0; it < SLOTS; ++it)
      vv[it] = ((unsigned)rown[it] < (unsigned)N) ? *reinterpret_cast<const uint4*>(Vb + (int64_t)rown[it] * sV_n)
                                                 : make_uint4(0, 0, 0, 0);
  }
  __syncthreads();
  // chunk max per head (each wavefront reduces its 32 rows)
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float mval = (lane < RPW) ? lg_s[g][wid * RPW + lane] : -INFINITY;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) mval = fmaxf(mval, __shfl_xor(mval, off, 64));
    if (lane == 0) red_s[g][wid] = mval;
  }
  __syncthreads();
  float mx[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    mx[g] = fmaxf(fmaxf(red_s[g][0], red_s[g][1]), fmaxf(red_s[g][2], red_s[g][3]));
    float p = 0.f;
    if (lane < RPW) {
      const float lgv = lg_s[g][wid * RPW + lane];
      p = (lgv == -INFINITY) ? 0.f : exp2f(lgv - mx[g]);
      lg_s[g][wid * RPW + lane] = p;
    }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) p += __shfl_xor(p, off, 64);
    if (lane == 0) sum_s[g][wid] = p;
  }
  __syncthreads();
  // weighted sum of this lane's V rows
  float o[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[g][e] = 0.f;
#pragma unroll
  for (int it = 0; it < SLOTS; ++it) {
    float vf[8];
    unpack8(vv[it], vf);
    const int r = it * 4 + rsub;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float p = lg_s[g][wid * RPW + r];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[g][e] = fmaf(p, vf[e], o[g][e]);
    }
  }
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
  float* pb = part + ((size_t)bh * nchunks + chunk) * G * (kHeadDim + 2);
  for (int e = threadIdx.x; e < G * kHeadDim; e += kAttnThreads) {
    const int g = e >> 7, d = e & 127;
    pb[g * (kHeadDim + 2) + 2 + d] = (o_s[0][g][d] + o_s[1][g][d]) + (o_s[2][g][d] + o_s[3][g][d]);
  }
  if (threadIdx.x < G) {
    const int g = threadIdx.x;
    pb[g * (kHeadDim + 2) + 0] = fmaxf(fmaxf(red_s[g][0], red_s[g][1]), fmaxf(red_s[g][2], red_s[g][3]));
    pb[g * (kHeadDim + 2) + 1] = (sum_s[g][0] + sum_s[g][1]) + (sum_s[g][2] + sum_s[g][3]);
  }

}

// ---------------------------------------------------------------------------
// 6. merge -- one workgroup per (b, query head): log-sum-exp combination of
// the chunk partials.  A separate launch (rather than a last-workgroup
// merge inside the attention kernel) because making the partials visible
// across the chip from inside a kernel needs a device-scope release per
// workgroup, which writes back the whole L2 of its XCD.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kHeadDim) void merge_kernel(int Hkv, int G, int nchunks, const float* __restrict__ part,
                                                         float* __restrict__ out) {
  const int bq = blockIdx.x;  // b * Hq + query head
  const int Hq = Hkv * G;
  const int b = bq / Hq, jq = bq % Hq;
  const int h = jq / G, g = jq % G;
  const size_t bh = (size_t)b * Hkv + h;
  const size_t cstride = (size_t)G * (kHeadDim + 2);
  const float* pg = part + bh * nchunks * cstride + (size_t)g * (kHeadDim + 2);
  __shared__ float w_s[1024];
  // global maximum over the chunks, then the weights, 1024 chunks per pass
  float Mx = -INFINITY;
  for (int t = 0; t < nchunks; ++t) Mx = fmaxf(Mx, pg[t * cstride]);
  float acc = 0.f, lsum = 0.f;
  for (int t0 = 0; t0 < nchunks; t0 += 1024) {
    const int nc = min(1024, nchunks - t0);
    for (int t = threadIdx.x; t < nc; t += kHeadDim) w_s[t] = exp2f(pg[(t0 + t) * cstride] - Mx);
    __syncthreads();
#pragma unroll 8
    for (int t = 0; t < nc; ++t) {
      lsum = fmaf(pg[(t0 + t) * cstride + 1], w_s[t], lsum);
      acc = fmaf(pg[(t0 + t) * cstride + 2 + threadIdx.x], w_s[t], acc);
    }
    __syncthreads();
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
  uint32_t* hist_fine = reinterpret_cast<uint32_t*>(a.ws + lay.off_hist_fine);
  uint32_t* hist_cc = reinterpret_cast<uint32_t*>(a.ws + lay.off_hist_cc);
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
                                                                hist_cc, a.score_out);
  mark(2);
  threshold_kernel<L><<<BH, 256, 0, st>>>(a.k, lay.nslices, hist_fine, hist_cc, sel_info, sel_base, tie_base);
  mark(3);
  select_kernel<<<dim3(lay.nslices, BH), kSelectThreads, 0, st>>>(a.k, lay.nslices, cand, cand_count, sel_info,
                                                                  sel_base, tie_base, idx);
  mark(4);
  const float scale_log2 = a.sm_scale * 1.4426950408889634f;
  const dim3 agrid(lay.nchunks, BH);
  switch (lay.G) {
#define BPC_ATTEND_CASE(GG)                                                                                     \
  case GG:                                                                                                      \
    attend_kernel<GG><<<agrid, kAttnThreads, 0, st>>>(a.N, a.k, a.Hkv, lay.nchunks, idx, a.q, a.K, a.sK_b,       \
                                                      a.sK_h, a.sK_n, a.V, a.sV_b, a.sV_h, a.sV_n, scale_log2,    \
                                                      part);                                                    \
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
