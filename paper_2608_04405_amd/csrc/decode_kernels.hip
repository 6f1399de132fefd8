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
//   3 select     per slice: the global k-th smallest distance T*, the number of ties at T*
//                that are taken, the slice's offset, and its selected keys (ascending key
//                order; ties at T* go to the lowest indices)
//   4 attend     per 128 selected keys: gather the K/V rows, softmax partials in fp32
//   5 merge      per query head: log-sum-exp merge of the partials
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
constexpr int kQpackThreads = 1024;

template <int L>
__global__ __launch_bounds__(kQpackThreads) void qpack_kernel(const uint16_t* __restrict__ q, const float* __restrict__ P,
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
    constexpr int PV = L * kHeadDim / 4 / kQpackThreads;  // float4 per thread
    float4 pv[PV];
#pragma unroll
    for (int r = 0; r < PV; ++r) pv[r] = reinterpret_cast<const float4*>(Pb)[r * kQpackThreads + threadIdx.x];
    const bool has_q = threadIdx.x < G * kHeadDim / 8;
    const uint4 qv = has_q ? reinterpret_cast<const uint4*>(qb)[threadIdx.x] : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int r = 0; r < PV; ++r) {
      const int e = 4 * (r * kQpackThreads + threadIdx.x);
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
  for (int base = 0; base < ntriples; base += kQpackThreads) {
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
// Each thread scores 16 keys (16-byte non-temporal loads, all issued before
// the first is consumed) and keeps their distances in registers; the slice
// histogram lives in LDS; the ordered candidate list is compacted with
// wavefront ballots.
// ---------------------------------------------------------------------------
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

template <int L>
struct ScanShared {
  static constexpr int NB = dist_bins(L);
  static constexpr int NBP = (NB + 127) & ~127;  // histogram padded to whole coarse bins
  uint32_t hist[NBP];
  uint32_t coarse[kCoarseBins];
  uint32_t cc[kCoarseBins + 1];
  int cnt[256];
  int cs, kth, total;
};

// FULL: the slice holds kSlice keys, so no per-key bounds tests are needed
template <int L, bool FULL>
__device__ __forceinline__ void scan_body(ScanShared<L>& sh, const uint32_t* __restrict__ codes, int64_t sC_b,
                                          int64_t sC_h, int Hkv, int N, int k, int nslices,
                                          const uint32_t* __restrict__ qcode_ws, const int* __restrict__ T_ws,
                                          uint32_t* __restrict__ cand, int* __restrict__ cand_count,
                                          uint32_t* __restrict__ hist_fine, uint32_t* __restrict__ hist_cc,
                                          int32_t* __restrict__ score_out) {
  constexpr int W = L / 32;
  constexpr int NB = ScanShared<L>::NB;
  constexpr int NBP = ScanShared<L>::NBP;
  constexpr int PER = kSlice / kScanThreads;  // keys per thread
  constexpr int KPL = 4 / W;                  // keys per 16-byte load
  constexpr int NLD = PER / KPL;              // loads per thread
  constexpr int KSTEP = kScanThreads * KPL;   // keys per load round of the workgroup
  constexpr int NW = kScanThreads / 64;
  static_assert(NLD * NW <= 256, "compaction offsets are scanned by one wavefront");
  uint32_t* hist_s = sh.hist;
  uint32_t* coarse_s = sh.coarse;
  uint32_t* cc_s = sh.cc;
  int* cnt_s = sh.cnt;
  int& cs_s = sh.cs;
  int& kth_sh = sh.kth;
  int& total_s = sh.total;

  const int s = blockIdx.x, bh = blockIdx.y;
  const int b = bh / Hkv, h = bh % Hkv;
  const int n0 = s * kSlice;
  const int cnt = min(kSlice, N - n0);
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;

  uint32_t sg[W], M[7][W];
  const uint32_t* qc = qcode_ws + (size_t)bh * 8 * W;
#pragma unroll
  for (int w = 0; w < W; ++w) {
    sg[w] = qc[w];
#pragma unroll
    for (int j = 0; j < 7; ++j) M[j][w] = qc[(1 + j) * W + w];
  }
#pragma unroll
  for (int r = 0; r < NBP / kScanThreads; ++r) hist_s[r * kScanThreads + threadIdx.x] = 0u;
  __syncthreads();

  const uint32_t* cb = codes + b * sC_b + h * sC_h + (int64_t)n0 * W;
  constexpr bool full = FULL;
  // a head's codes are W-word aligned; 16-byte loads need a 16-byte aligned base
  const bool vec_ok = (reinterpret_cast<uintptr_t>(cb) & 15u) == 0;
  // two rounds of NLD / 2 loads: every load of a round is issued before the
  // first is consumed, and at most half of the thread's codes are live
  constexpr int HALF = NLD / 2;
  // distances (< 2^14) packed two per register: key i = it * KPL + u is half i & 1 of dpk[i >> 1]
  uint32_t dpk[PER / 2];
#pragma unroll
  for (int round = 0; round < 2; ++round) {
    u32x4_t cw[HALF];
    if (vec_ok) {
      // groups that reach past the slice's last key re-read group 0 (their
      // keys are masked out below)
#pragma unroll
      for (int r = 0; r < HALF; ++r) {
        const int n = (round * HALF + r) * KSTEP + threadIdx.x * KPL;
        const int nl = (full || n + KPL <= cnt) ? n : 0;
        cw[r] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(cb + (int64_t)nl * W));
      }
    } else {
      for (int r = 0; r < HALF; ++r) {
        const int n = (round * HALF + r) * KSTEP + threadIdx.x * KPL;
        uint32_t t4[4] = {0u, 0u, 0u, 0u};
        for (int u = 0; u < KPL; ++u)
          if (n + u < cnt)
            for (int w = 0; w < W; ++w) t4[u * W + w] = cb[(int64_t)(n + u) * W + w];
        cw[r] = u32x4_t{t4[0], t4[1], t4[2], t4[3]};
      }
    }
#pragma unroll
    for (int r = 0; r < HALF; ++r) {
      const int it = round * HALF + r;
#pragma unroll
      for (int u = 0; u < KPL; ++u) {
        uint32_t d = 0;
#pragma unroll
        for (int j = 0; j < 7; ++j) {
          uint32_t pc = 0;
#pragma unroll
          for (int w = 0; w < W; ++w) pc += __popc(M[j][w] & (cw[r][u * W + w] ^ sg[w]));
          d += pc << j;
        }
        const int i = it * KPL + u;
        dpk[i >> 1] = (i & 1) ? (dpk[i >> 1] | (d << 16)) : d;
        if (full || it * KSTEP + threadIdx.x * KPL + u < cnt) atomicAdd(&hist_s[d], 1u);
      }
    }
  }
  __syncthreads();
  auto dist_of = [&](int it, int u) -> int {
    const int i = it * KPL + u;
    return (int)((dpk[i >> 1] >> ((i & 1) << 4)) & 0xFFFFu);
  };
  auto is_cand = [&](int it, int u, int kth) -> bool {
    return (full || it * KSTEP + threadIdx.x * KPL + u < cnt) && dist_of(it, u) <= kth;
  };

  // eight threads per coarse bin, sixteen fine bins each: counts and the
  // prefix within the coarse bin
  const int cbin = threadIdx.x >> 3, part = threadIdx.x & 7;
  const int fb0 = (cbin << kCoarseShift) + part * 16;
  uint32_t cntv[16];
  int local = 0;
  if (fb0 < NBP) {
    const uint4* hv = reinterpret_cast<const uint4*>(hist_s + fb0);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const uint4 x = hv[r];
      cntv[4 * r] = x.x, cntv[4 * r + 1] = x.y, cntv[4 * r + 2] = x.z, cntv[4 * r + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int e = 0; e < 16; ++e) cntv[e] = 0u;
  }
#pragma unroll
  for (int e = 0; e < 16; ++e) local += (int)cntv[e];
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

  // candidates (dist <= kth) in key order; key n = it * KSTEP + t * KPL + u,
  // so the order is (it, wavefront, lane, u).  Pass 1 counts per (it,
  // wavefront), one wavefront scans the counts, pass 2 writes.
#pragma unroll
  for (int it = 0; it < NLD; ++it) {
    int c = 0;
#pragma unroll
    for (int u = 0; u < KPL; ++u) c += __popcll(__ballot(is_cand(it, u, kth)));
    if (lane == 0) cnt_s[it * NW + wid] = c;
  }
  __syncthreads();
  if (threadIdx.x < 64) {
    // exclusive prefix over the (it, wavefront) counts, four per lane
    int v[4], tot = 0;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 4 * lane + r;
      v[r] = (i < NLD * NW) ? cnt_s[i] : 0;
      tot += v[r];
    }
    int x = tot;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    int run = x - tot;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 4 * lane + r;
      if (i < NLD * NW) cnt_s[i] = run;
      run += v[r];
    }
    if (lane == 63) total_s = x;
  }
  __syncthreads();
  uint32_t* cs_out = cand + sl * kSlice;
#pragma unroll
  for (int it = 0; it < NLD; ++it) {
    int pos = cnt_s[it * NW + wid];
    bool f[KPL];
#pragma unroll
    for (int u = 0; u < KPL; ++u) {
      f[u] = is_cand(it, u, kth);
      const unsigned long long m = __ballot(f[u]);
      pos += (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    }
#pragma unroll
    for (int u = 0; u < KPL; ++u) {
      if (f[u]) {
        const int n = it * KSTEP + threadIdx.x * KPL + u;
        cs_out[pos++] = ((uint32_t)n << 16) | (uint32_t)dist_of(it, u);
      }
    }
  }
  if (threadIdx.x == 0) cand_count[sl] = total_s;
  if (score_out) {  // debug output
    const int T = T_ws[bh];
    int32_t* so = score_out + (size_t)bh * N + n0;
#pragma unroll
    for (int it = 0; it < NLD; ++it)
#pragma unroll
      for (int u = 0; u < KPL; ++u) {
        const int n = it * KSTEP + threadIdx.x * KPL + u;
        if (n < cnt) so[n] = T - 2 * dist_of(it, u);
      }
  }
}

// two 1024-thread workgroups per CU (8 wavefronts per SIMD) let one
// workgroup stream codes while the other runs its histogram phases
template <int L>
__global__ __launch_bounds__(kScanThreads) __attribute__((amdgpu_waves_per_eu(L <= 64 ? 8 : 4))) void scan_kernel(
    const uint32_t* __restrict__ codes, int64_t sC_b, int64_t sC_h, int Hkv, int N, int k, int nslices,
    const uint32_t* __restrict__ qcode_ws, const int* __restrict__ T_ws, uint32_t* __restrict__ cand,
    int* __restrict__ cand_count, uint32_t* __restrict__ hist_fine, uint32_t* __restrict__ hist_cc,
    int32_t* __restrict__ score_out) {
  __shared__ ScanShared<L> sh;
  if ((int)(blockIdx.x + 1) * kSlice <= N)
    scan_body<L, true>(sh, codes, sC_b, sC_h, Hkv, N, k, nslices, qcode_ws, T_ws, cand, cand_count, hist_fine,
                       hist_cc, score_out);
  else
    scan_body<L, false>(sh, codes, sC_b, sC_h, Hkv, N, k, nslices, qcode_ws, T_ws, cand, cand_count, hist_fine,
                        hist_cc, score_out);
}

// ---------------------------------------------------------------------------
// 3. select -- one workgroup per slice.  From the prefix-form histograms of
// all slices of its (b, h) it derives the global threshold T* (the k-th
// smallest distance), the number of keys at T* that are taken (lowest
// indices first) and its own output offset, then writes its selected keys
// in ascending key order.  The slice's candidate loads are issued first, so
// they are in flight while the threshold is derived.
// ---------------------------------------------------------------------------
template <int L>
__global__ __launch_bounds__(kSelectThreads) void select_kernel(int k, int nslices, const uint32_t* __restrict__ cand,
                                                               const int* __restrict__ cand_count,
                                                               const uint32_t* __restrict__ hist_fine,
                                                               const uint32_t* __restrict__ hist_cc,
                                                               int32_t* __restrict__ idx) {
  constexpr int NB = dist_bins(L);
  constexpr int FS = fine_stride(L);
  constexpr int PER = 16;
  constexpr int NWV = kSelectThreads / 64;
  __shared__ int wave_tot[NWV];
  __shared__ int gp_s[kCoarseBins];
  __shared__ int fe_s[1 << kCoarseShift];
  __shared__ int first_s[2];
  __shared__ int red_s[2][NWV];
  const int s = blockIdx.x, bh = blockIdx.y;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const size_t sl = (size_t)bh * nslices + s;
  const int cnt = cand_count[sl];
  const uint32_t* cs = cand + sl * kSlice;

  // first batch of candidates (16 per thread), in flight during the threshold
  uint32_t cv[PER];
  auto load_batch = [&](int base) {
    const int i0 = base + threadIdx.x * PER;
    if (i0 + PER <= cnt) {
      const uint4* v = reinterpret_cast<const uint4*>(cs + i0);
#pragma unroll
      for (int r = 0; r < PER / 4; ++r) {
        const uint4 x = v[r];
        cv[4 * r] = x.x, cv[4 * r + 1] = x.y, cv[4 * r + 2] = x.z, cv[4 * r + 3] = x.w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < PER; ++e) cv[e] = (i0 + e < cnt) ? cs[i0 + e] : 0xFFFFFFFFu;  // 0xFFFF > any T*
    }
  };
  load_batch(0);

  // ---- global threshold of this (b, h)
  const uint32_t* ccb = hist_cc + (size_t)bh * nslices * kCoarseStride;
  const uint32_t* hfb = hist_fine + (size_t)bh * nslices * FS;
  if (threadIdx.x < kCoarseBins) {
    // GP(c + 1): keys of all slices with distance < 128 (c + 1)
    int acc = 0;
#pragma unroll 8
    for (int t = 0; t < nslices; ++t) acc += (int)ccb[(size_t)t * kCoarseStride + threadIdx.x + 1];
    gp_s[threadIdx.x] = acc;
    const unsigned long long m = __ballot(acc >= k);
    if (lane == 0) first_s[wid] = m ? first_lane(m) + 64 * wid : (1 << 30);
  }
  __syncthreads();
  const int cstar = min(min(first_s[0], first_s[1]), kCoarseBins - 1);
  const int below_c = (cstar > 0) ? gp_s[cstar - 1] : 0;
  __syncthreads();
  if (threadIdx.x < (1 << kCoarseShift)) {
    // fine bins of C*: inclusive prefix within the coarse bin, over all slices
    // (bins above T* may be stale in some slices; only bins up to T* are used)
    const int t = (cstar << kCoarseShift) + threadIdx.x;
    int inc = 0, exc = 0;
    if (t < NB) {
#pragma unroll 8
      for (int u = 0; u < nslices; ++u) {
        const uint32_t v = hfb[(size_t)u * FS + t];
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
  const int quota = k - (below_c + fe_s[tt]);
  // keys below T* and ties at T* in the slices before this one
  int bl = 0, ti = 0;
  for (int u = threadIdx.x; u < s; u += kSelectThreads) {
    const uint32_t v = hfb[(size_t)u * FS + tstar];
    bl += (int)ccb[(size_t)u * kCoarseStride + cstar] + (int)(v >> 16);
    ti += (int)(v & 0xFFFFu);
  }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    bl += __shfl_xor(bl, o, 64);
    ti += __shfl_xor(ti, o, 64);
  }
  if (lane == 0) red_s[0][wid] = bl, red_s[1][wid] = ti;
  __syncthreads();
  int below_before = 0, ties_before = 0;
#pragma unroll
  for (int w = 0; w < NWV; ++w) below_before += red_s[0][w], ties_before += red_s[1][w];
  int out_pos = below_before + min(ties_before, quota);

  // ---- ordered selection
  int32_t* ib = idx + (size_t)bh * k;
  const int n0 = s * kSlice;
  for (int base = 0; base < cnt; base += kSelectThreads * PER) {
    if (base > 0) load_batch(base);
    int nb = 0, nt = 0;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int d = (int)(cv[e] & 0xFFFFu);
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
    const int tb = tot & 0xFFFF, tt2 = tot >> 16;
    out_pos += tb + max(0, min(ties_before + tt2, quota) - min(ties_before, quota));
    ties_before += tt2;
  }
}

// ---------------------------------------------------------------------------
// 4. attention over the selected rows -- one workgroup per 128 selected keys
// Sixteen lanes share a key row (lane l16 holds dims [8 l16, 8 l16 + 8)),
// four rows per wavefront instruction, 32 rows per wavefront; the wavefront
// loads its 32 row indices once and issues every K and V row load before
// the first is consumed.  Logits are kept in base 2 (sm_scale * log2 e).
// Each workgroup writes one (max, sum, weighted V) partial per query head.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// a + (bf16 pair x) . (bf16 pair y), fp32 accumulation
__device__ __forceinline__ float dot2_bf16(uint32_t x, uint32_t y, float a) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, x), __builtin_bit_cast(bf16x2_t, y), a, false);
}

// sum over each row of 16 lanes, every lane of the row receives it (DPP:
// swap neighbours, swap pairs, mirror within 8, mirror within 16)
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_f32<0xB1>(v);
  v += dpp_f32<0x4E>(v);
  v += dpp_f32<0x141>(v);
  v += dpp_f32<0x140>(v);
  return v;
}

__device__ __forceinline__ void unpack8(const uint4 v, float (&f)[8]) {
  f[0] = bf16_to_f32(v.x & 0xFFFFu), f[1] = bf16_to_f32(v.x >> 16);
  f[2] = bf16_to_f32(v.y & 0xFFFFu), f[3] = bf16_to_f32(v.y >> 16);
  f[4] = bf16_to_f32(v.z & 0xFFFFu), f[5] = bf16_to_f32(v.z >> 16);
  f[6] = bf16_to_f32(v.w & 0xFFFFu), f[7] = bf16_to_f32(v.w >> 16);
}

// max / sum over lanes [0, 32) of a wavefront; every lane receives it
__device__ __forceinline__ float wave32_max(float v) {
  v = fmaxf(v, dpp_f32<0xB1>(v));
  v = fmaxf(v, dpp_f32<0x4E>(v));
  v = fmaxf(v, dpp_f32<0x141>(v));
  v = fmaxf(v, dpp_f32<0x140>(v));
  return fmaxf(v, __shfl_xor(v, 16, 64));
}
__device__ __forceinline__ float wave32_sum(float v) {
  v = row16_sum(v);
  return v + __shfl_xor(v, 16, 64);
}

// One chunk of selected rows.  FULL: all kAttnChunk rows are valid, so the
// loads need no bounds checks (every chunk but the last of a (b, h)).
template <int G, bool FULL>
__device__ __forceinline__ void attend_chunk(int N, int k, int chunk, int bh, int b, int h, int Hkv,
                                             const int32_t* __restrict__ idx, const uint16_t* __restrict__ q,
                                             const char* Kh, uint32_t kstride, const char* Vh, uint32_t vstride,
                                             float scale_log2, float* __restrict__ pb, float (*lg_s)[kAttnChunk],
                                             float (*red_s)[4], float (*sum_s)[4], float (*o_s)[G][kHeadDim]) {
  constexpr int RPW = kAttnChunk / (kAttnThreads / 64);  // rows per wavefront (32)
  constexpr int SLOTS = RPW / 4;                          // rows per lane (8)
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int l16 = lane & 15, rsub = lane >> 4;
  const int j0 = chunk * kAttnChunk + wid * RPW;  // first selected row of this wavefront
  const int nrows = FULL ? RPW : max(0, min(RPW, k - j0));
  int myidx = 0;
  if (FULL || lane < nrows) myidx = idx[(size_t)bh * k + j0 + (lane & (RPW - 1))];
  bool ok[SLOTS];
  uint32_t rown[SLOTS];
#pragma unroll
  for (int it = 0; it < SLOTS; ++it) {
    const int n = __shfl(myidx, it * 4 + rsub, 64);
    ok[it] = FULL ? true : ((it * 4 + rsub < nrows) && (unsigned)n < (unsigned)N);
    rown[it] = ok[it] ? (uint32_t)n : 0u;  // row 0 of the head always exists
  }
  uint4 kv[SLOTS], vv[SLOTS];
#pragma unroll
  for (int it = 0; it < SLOTS; ++it) kv[it] = *reinterpret_cast<const uint4*>(Kh + (rown[it] * kstride + 16u * l16));
  if constexpr (G <= 4) {
#pragma unroll
    for (int it = 0; it < SLOTS; ++it)
      vv[it] = *reinterpret_cast<const uint4*>(Vh + (rown[it] * vstride + 16u * l16));
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
      if (l16 == 0) lg_s[g][wid * RPW + r] = ok[it] ? a * scale_log2 : -INFINITY;
    }
  }
  if constexpr (G > 4) {
#pragma unroll
    for (int it = 0; it < SLOTS; ++it)
      vv[it] = *reinterpret_cast<const uint4*>(Vh + (rown[it] * vstride + 16u * l16));
  }
  __syncthreads();
  // chunk max per head (each wavefront reduces its 32 rows)
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const float mval = wave32_max(lg_s[g][wid * RPW + (lane & (RPW - 1))]);
    if (lane == 0) red_s[g][wid] = mval;
  }
  __syncthreads();
  float mx[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    mx[g] = fmaxf(fmaxf(red_s[g][0], red_s[g][1]), fmaxf(red_s[g][2], red_s[g][3]));
    const float lgv = lg_s[g][wid * RPW + (lane & (RPW - 1))];
    float p = (lgv == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(lgv - mx[g]);
    const float tot = wave32_sum(lane < RPW ? p : 0.f);
    if (lane < RPW) lg_s[g][wid * RPW + lane] = p;
    if (lane == 0) sum_s[g][wid] = tot;
  }
  __syncthreads();
  // weighted sum of this lane's V rows (rows that are not selected have p = 0
  // and contribute nothing: their V load reads row 0, which is zeroed here)
  float o[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[g][e] = 0.f;
#pragma unroll
  for (int it = 0; it < SLOTS; ++it) {
    uint4 v = vv[it];
    if (!FULL && !ok[it]) v = make_uint4(0, 0, 0, 0);
    float vf[8];
    unpack8(v, vf);
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
  for (int e = threadIdx.x; e < G * kHeadDim; e += kAttnThreads) {
    const int g = e >> 7, d = e & 127;
    pb[g * (kHeadDim + 2) + 2 + d] = (o_s[0][g][d] + o_s[1][g][d]) + (o_s[2][g][d] + o_s[3][g][d]);
  }
  if (threadIdx.x < G) {
    const int g = threadIdx.x;
    pb[g * (kHeadDim + 2) + 0] = mx[g];
    pb[g * (kHeadDim + 2) + 1] = (sum_s[g][0] + sum_s[g][1]) + (sum_s[g][2] + sum_s[g][3]);
  }
}

template <int G>
__global__ __launch_bounds__(kAttnThreads) void attend_kernel(
    int N, int k, int Hkv, int nchunks, const int32_t* __restrict__ idx, const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ K, int64_t sK_b, int64_t sK_h, int64_t sK_n, const uint16_t* __restrict__ V,
    int64_t sV_b, int64_t sV_h, int64_t sV_n, float scale_log2, float* __restrict__ part) {
  __shared__ float lg_s[G][kAttnChunk];
  __shared__ float red_s[G][4];
  __shared__ float sum_s[G][4];
  __shared__ float o_s[4][G][kHeadDim];
  const int chunk = blockIdx.x, bh = blockIdx.y;
  const int b = bh / Hkv, h = bh % Hkv;
  // head bases are uniform; a row's byte offset within its head fits 32 bits
  const char* Kh = reinterpret_cast<const char*>(K + b * sK_b + h * sK_h);
  const char* Vh = reinterpret_cast<const char*>(V + b * sV_b + h * sV_h);
  float* pb = part + ((size_t)bh * nchunks + chunk) * G * (kHeadDim + 2);
  if ((chunk + 1) * kAttnChunk <= k)
    attend_chunk<G, true>(N, k, chunk, bh, b, h, Hkv, idx, q, Kh, (uint32_t)sK_n * 2u, Vh, (uint32_t)sV_n * 2u,
                          scale_log2, pb, lg_s, red_s, sum_s, o_s);
  else
    attend_chunk<G, false>(N, k, chunk, bh, b, h, Hkv, idx, q, Kh, (uint32_t)sK_n * 2u, Vh, (uint32_t)sV_n * 2u,
                           scale_log2, pb, lg_s, red_s, sum_s, o_s);
}

// ---------------------------------------------------------------------------
// 5. merge -- one workgroup per (b, query head): log-sum-exp combination of
// the chunk partials.  A separate launch (rather than a last-workgroup
// merge inside the attention kernel) because making the partials visible
// across the chip from inside a kernel needs a device-scope release per
// workgroup, which writes back the whole L2 of its XCD.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kHeadDim) void merge_kernel(int Hkv, int G, int nchunks, const float* __restrict__ part,
                                                         float* __restrict__ out) {
  constexpr int CB = 512;  // chunks per pass
  const int bq = blockIdx.x;  // b * Hq + query head
  const int Hq = Hkv * G;
  const int b = bq / Hq, jq = bq % Hq;
  const int h = jq / G, g = jq % G;
  const size_t bh = (size_t)b * Hkv + h;
  const size_t cstride = (size_t)G * (kHeadDim + 2);
  const float* pg = part + bh * nchunks * cstride + (size_t)g * (kHeadDim + 2);
  __shared__ float m_s[CB], l_s[CB];
  __shared__ float mx_s[2];
  // global maximum: the chunk maxima are loaded in parallel
  float mloc = -INFINITY;
  for (int t = threadIdx.x; t < nchunks; t += kHeadDim) mloc = fmaxf(mloc, pg[t * cstride]);
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) mloc = fmaxf(mloc, __shfl_xor(mloc, o, 64));
  if ((threadIdx.x & 63) == 0) mx_s[threadIdx.x >> 6] = mloc;
  __syncthreads();
  const float Mx = fmaxf(mx_s[0], mx_s[1]);
  float acc = 0.f, lsum = 0.f;
  for (int t0 = 0; t0 < nchunks; t0 += CB) {
    const int nc = min(CB, nchunks - t0);
    for (int t = threadIdx.x; t < nc; t += kHeadDim) {
      m_s[t] = exp2f(pg[(t0 + t) * cstride] - Mx);
      l_s[t] = pg[(t0 + t) * cstride + 1];
    }
    __syncthreads();
#pragma unroll 8
    for (int t = 0; t < nc; ++t) {
      lsum = fmaf(l_s[t], m_s[t], lsum);
      acc = fmaf(pg[(t0 + t) * cstride + 2 + threadIdx.x], m_s[t], acc);
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
  int32_t* idx = a.idx_out ? a.idx_out : reinterpret_cast<int32_t*>(a.ws + lay.off_idx);
  float* part = reinterpret_cast<float*>(a.ws + lay.off_part);
  hipStream_t st = a.stream;
  auto mark = [&](int i) {
    if (a.events) (void)hipEventRecord(a.events[i], st);
  };

  mark(0);
  qpack_kernel<L><<<BH, kQpackThreads, 0, st>>>(a.q, a.P, a.sP_b, a.sP_h, a.Hkv, lay.G, qcode, T, a.qcode_out);
  mark(1);
  scan_kernel<L><<<dim3(lay.nslices, BH), kScanThreads, 0, st>>>(a.codes, a.sC_b, a.sC_h, a.Hkv, a.N, a.k,
                                                                lay.nslices, qcode, T, cand, cand_count, hist_fine,
                                                                hist_cc, a.score_out);
  mark(2);
  select_kernel<L><<<dim3(lay.nslices, BH), kSelectThreads, 0, st>>>(a.k, lay.nslices, cand, cand_count, hist_fine,
                                                                     hist_cc, idx);
  mark(3);
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
  mark(4);
  merge_kernel<<<a.B * a.Hq, kHeadDim, 0, st>>>(a.Hkv, lay.G, lay.nchunks, part, a.out);
  mark(5);
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
