// Decode-step kernels: query packing, XOR/popcount scoring, exact top-k
// selection and sparse attention over the gathered K/V rows (Sec. 3.2
// "Retrieval Phase"; Algorithm "Computing hashing score"; Appendix "CUDA
// Optimizations on Bitwise Operations"; Sec. 4.2 "Kernel Evaluation").
//
// Selection works on the weighted Hamming distance
//     dist_n = sum_j 2^j popcount(M_j & (code_n XOR s)),   c_n = sum|p| - 2 dist_n,
// so the k largest scores are the k smallest distances, and distances are
// small integers in [0, 127 L].  A (sequence b, KV head h) is cut into slices
// of kSlice consecutive keys.  Three launches per step:
//   1 score   one workgroup per slice: projects, quantises and packs the query
//             group (every slice of (b, h) does it; they share an XCD, so P
//             comes from HBM once), scores the slice's codes into an LDS
//             histogram, finds the slice's own k-th smallest distance kth_s,
//             and writes its histograms up to kth_s, a window record of
//             cumulative counts around its share of the threshold, and its
//             candidates (dist <= cand_max <= kth_s) in key order.
//   2 attend  one workgroup per slice: from the histograms of every slice of
//             (b, h) it derives the global k-th smallest distance T*, how
//             many keys at T* its slice keeps (lowest indices first) and its
//             output offset; it keeps those candidates (ascending key order),
//             writes their indices, gathers their K/V rows and accumulates
//             softmax partials in fp32.
//   3 merge   per query head: log-sum-exp merge of the slices' partials.
// T* is never above any slice's kth_s (that slice alone already holds k keys
// at or below kth_s, or all of its keys when it has fewer than k), so the
// candidates contain every selected key and every histogram bin at or below
// T* is written by every slice.

#include <atomic>

#include "bpc_internal.h"

namespace bpc {

// ---------------------------------------------------------------------------
// Phase trace (only in builds with -DBPC_TRACE; the product build has none):
// thread 0 of each workgroup stores the 100 MHz real-time counter at the
// phase boundaries of its kernel into trace[(kernel * 65536 + workgroup) * 16
// + slot] (slots 0..11), and a value of its own with BPC_NOTE (slots 12..15;
// slot 15 = the XCC the workgroup ran on), in a buffer the host registers
// with bpc_trace_buffer().
// ---------------------------------------------------------------------------
#ifdef BPC_TRACE
__device__ unsigned long long* g_trace = nullptr;
#define BPC_NOTE(kern, slot, val)                                                                \
  do {                                                                                           \
    if (threadIdx.x == 0 && g_trace && blockIdx.x < 65536)                                       \
      g_trace[((size_t)(kern) * 65536 + blockIdx.x) * 16 + (slot)] = (unsigned long long)(val); \
  } while (0)
// hwreg(HW_REG_XCC_ID): bits 3:0 = the XCC of this wavefront
#define BPC_STAMP(kern, slot)                                                                 \
  do {                                                                                        \
    BPC_NOTE(kern, slot, __builtin_amdgcn_s_memrealtime());                                   \
    if ((slot) == 0) BPC_NOTE(kern, 15, __builtin_amdgcn_s_getreg((3 << 11) | 20) & 15);      \
    if ((slot) == 0) BPC_NOTE(kern, 11, __builtin_amdgcn_s_getreg((31 << 11) | 4));          \
  } while (0)
#else
#define BPC_STAMP(kern, slot) ((void)0)
#define BPC_NOTE(kern, slot, val) ((void)0)
#endif

// Workgroup id -> (b, h) and slice.  Workgroups are dispatched to the eight
// XCDs round-robin by id; all slices of one (b, h) get ids with the same
// residue mod 8, so they run on one XCD and share its L2 (P, q, candidates).
__device__ __forceinline__ void slice_tile(int id, int BH, int nslices, int& bh, int& s) {
  const int grp = id / (8 * nslices);
  const int r = id - grp * 8 * nslices;
  const int m = min(8, BH - grp * 8);  // (b, h) pairs in this group of eight
  // the divisions run on the vector unit: mark the results as uniform so that
  // everything addressed through them stays in scalar registers
  bh = __builtin_amdgcn_readfirstlane(grp * 8 + r % m);
  s = __builtin_amdgcn_readfirstlane(r / m);
}

// ---------------------------------------------------------------------------
// Query projection, quantisation and packing (Sec. 3.2 "Retrieval Phase";
// Appendix "Packing kernel"), done by every scoring workgroup for its own
// (b, h) before its code stream starts (one code load per thread goes out
// behind the P loads), so that the loads of P and q are not queued behind
// the code stream of other workgroups.  All slices of a
// (b, h) run on one XCD: P and q come from HBM once, then from its L2.
//
// P is loaded with coalesced 16-byte loads and staged in LDS (in the place
// of the slice histogram), 16-byte unit r of block c = coordinates
// [32 c + 4 r, 32 c + 4 r + 4) of row i at i 32 + 8 c + (r ^ (c + 4 (i & 1))):
// the eight lanes (two rows x four blocks) that read one unit index at a
// time then hit eight different bank groups.  Thread t < 4 L owns block
// c = t mod 4 of row i = t / 4: for each query head g, in ascending order,
// it sums its 32 coordinates in ascending order from +0, the quad of lanes
// sharing i combines the block sums as ((b0 + b1) + (b2 + b3)), and the
// heads are added in ascending g.  Each product of a bf16 query coordinate
// and an fp32 entry of P is exact in fp64 (8 + 24 significant bits), so a
// fused multiply-add rounds exactly as the separately rounded multiply and
// add would.  The group sum is quantised to [-127, 127] (scale 127 / max |x|,
// rounded half away from zero) and packed into 1 sign + 7 magnitude planes.
// ---------------------------------------------------------------------------
template <int L, int GMAX = kMaxGroup>
struct QpackShared {
  float4 P[L * 32];             // P, 16-byte units in the swizzled order above
  uint4 q[GMAX][kHeadDim / 8];  // the group's queries, bf16 (at most GMAX heads)
};

// small per-workgroup state of the packing (kept outside the histogram)
template <int L>
struct QpackOut {
  double wmax[kScoreThreads / 64];  // max |xbar| per wavefront
  uint16_t qc16[8 * (L / 16)];      // the planes as 16-bit pieces (little-endian words of qc)
};

__device__ __forceinline__ int qpack_swz(int i, int c) { return c + 4 * (i & 1); }

// x of lane l ^ 1 and of lane l ^ 2 (DPP quad permutations), for doubles
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
  const int lo = __builtin_amdgcn_mov_dpp(__double2loint(x), CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_mov_dpp(__double2hiint(x), CTRL, 0xF, 0xF, false);
  return __hiloint2double(hi, lo);
}
constexpr int kDppQuadXor1 = 0xB1;    // quad_perm [1, 0, 3, 2]
constexpr int kDppQuadXor2 = 0x4E;    // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141;  // lane i <-> 7 - i within 8 lanes
constexpr int kDppMirror = 0x140;      // lane i <-> 15 - i within 16 lanes

// bit 4 k of m, for k = 0..15, packed into the low 16 bits
__device__ __forceinline__ uint32_t every_fourth_bit(unsigned long long m) {
  m &= 0x1111111111111111ull;
  m = (m | (m >> 3)) & 0x0303030303030303ull;
  m = (m | (m >> 6)) & 0x000F000F000F000Full;
  m = (m | (m >> 12)) & 0x000000FF000000FFull;
  m = (m | (m >> 24)) & 0x000000000000FFFFull;
  return (uint32_t)m;
}

// The planes land in o.qc16 (read them as 8 W little-endian u32 words: plane
// 0 = signs, plane 1 + j = bit j of |p|).  after_loads() runs right after
// the P and query loads are issued, so that the caller can put loads of its
// own in flight behind them.  Ends with a barrier; sh is free after it.
template <int L, int NT, int GMAX, class AfterLoads>
__device__ __forceinline__ void qpack_block(QpackShared<L, GMAX>& sh, QpackOut<L>& o, const uint16_t* __restrict__ qg,
                                            const float* __restrict__ Pbh, int G, AfterLoads&& after_loads) {
  static_assert((L * 32) % NT == 0 && NT % 64 == 0, "thread count");
  constexpr int PV = L * 32 / NT;                // 16-byte units of P per thread
  constexpr int RP = (4 * L + NT - 1) / NT;      // passes over the rows (a quad of lanes per row)
  constexpr int ACTW = (4 * L < NT ? 4 * L : NT) / 64;  // wavefronts holding rows
  const int t = threadIdx.x, lane = t & 63, wid = t >> 6;
  {
    float4 pv[PV];
#pragma unroll
    for (int r = 0; r < PV; ++r) pv[r] = reinterpret_cast<const float4*>(Pbh)[t + NT * r];
    uint4 qv[(GMAX * (kHeadDim / 8) + NT - 1) / NT];
#pragma unroll
    for (int r = 0; r < (GMAX * (kHeadDim / 8) + NT - 1) / NT; ++r) {
      const int e = t + NT * r;
      qv[r] = (e < G * (kHeadDim / 8)) ? reinterpret_cast<const uint4*>(qg)[e] : make_uint4(0u, 0u, 0u, 0u);
    }
    after_loads();
#pragma unroll
    for (int r = 0; r < PV; ++r) {
      const int f = t + NT * r;  // unit f of P: row f / 32, block (f / 8) mod 4, unit f mod 8
      const int i = f >> 5, c = (f >> 3) & 3, u = f & 7;
      sh.P[i * 32 + c * 8 + (u ^ qpack_swz(i, c))] = pv[r];
    }
#pragma unroll
    for (int r = 0; r < (GMAX * (kHeadDim / 8) + NT - 1) / NT; ++r) {
      const int e = t + NT * r;
      if (e < G * (kHeadDim / 8)) sh.q[e / (kHeadDim / 8)][e % (kHeadDim / 8)] = qv[r];
    }
  }
  __syncthreads();
  BPC_STAMP(1, 6);
  double xb[RP];  // the group sum of row (t + NT rr) / 4 (every lane of the quad)
  if (t < 4 * L) {  // whole wavefronts (4 L is a multiple of 64)
    double m = 0.0;
#pragma unroll
    for (int rr = 0; rr < RP; ++rr) {
      xb[rr] = 0.0;
      if (t + NT * rr >= 4 * L) continue;  // uniform over the wavefront
      const int i = (t + NT * rr) >> 2, c = t & 3;
      // four heads at a time: four independent fixed-order chains interleave;
      // P is re-read from LDS eight coordinates at a time (held whole, as 32
      // values, it would not fit beside the accumulators)
      for (int g0 = 0; g0 < G; g0 += 4) {
        double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll 1
        for (int j = 0; j < 4; ++j) {
          const float4 pa = sh.P[i * 32 + c * 8 + ((2 * j) ^ qpack_swz(i, c))];
          const float4 pb = sh.P[i * 32 + c * 8 + ((2 * j + 1) ^ qpack_swz(i, c))];
          const float pf[8] = {pa.x, pa.y, pa.z, pa.w, pb.x, pb.y, pb.z, pb.w};
          uint32_t w4[4][4];
#pragma unroll
          for (int hh = 0; hh < 4; ++hh) {
            // coordinates 32 c + 8 j .. 32 c + 8 j + 7 of head g0 + hh (a head
            // past G reads head g0, whose result is dropped)
            const uint4 qq = sh.q[g0 + hh < G ? (g0 + hh) % GMAX : g0 % GMAX][4 * c + j];
            w4[hh][0] = qq.x, w4[hh][1] = qq.y, w4[hh][2] = qq.z, w4[hh][3] = qq.w;
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const double d0 = (double)pf[2 * e], d1 = (double)pf[2 * e + 1];
#pragma unroll
            for (int hh = 0; hh < 4; ++hh) {
              acc[hh] = __builtin_fma(d0, (double)bf16_to_f32(w4[hh][e] & 0xFFFFu), acc[hh]);
              acc[hh] = __builtin_fma(d1, (double)bf16_to_f32(w4[hh][e] >> 16), acc[hh]);
            }
          }
        }
#pragma unroll
        for (int hh = 0; hh < 4; ++hh) {
          // ((b0 + b1) + (b2 + b3)) on every lane of the quad
          const double s01 = dadd(acc[hh], dpp_f64<kDppQuadXor1>(acc[hh]));
          const double a = dadd(s01, dpp_f64<kDppQuadXor2>(s01));
          if (g0 + hh < G) xb[rr] = (g0 + hh == 0) ? a : dadd(xb[rr], a);
        }
      }
      m = fmax(m, fabs(xb[rr]));
    }
    // max |xbar| of the wavefront: the quads are uniform, so two mirrors
    // give the maximum of 16 lanes, and four read-lanes that of the wavefront
    m = fmax(m, dpp_f64<kDppHalfMirror>(m));
    m = fmax(m, dpp_f64<kDppMirror>(m));
    const int mlo = __double2loint(m), mhi = __double2hiint(m);
    auto rl = [&](int l) {
      return __hiloint2double(__builtin_amdgcn_readlane(mhi, l), __builtin_amdgcn_readlane(mlo, l));
    };
    m = fmax(fmax(rl(0), rl(16)), fmax(rl(32), rl(48)));
    if (lane == 0) o.wmax[wid] = m;
  }
  __syncthreads();
  BPC_STAMP(1, 7);
  if (t < 4 * L) {
    double m = o.wmax[0];
#pragma unroll
    for (int w = 1; w < ACTW; ++w) m = fmax(m, o.wmax[w]);
#pragma unroll
    for (int rr = 0; rr < RP; ++rr) {
      if (t + NT * rr >= 4 * L) continue;
      const int p = (m > 0.0) ? (int)round(dmul(xb[rr], 127.0) / m) : 0;
      const uint32_t mag = (uint32_t)abs(p);
      // every quad holds one row: each plane's ballot has its bits at lanes 4 k
#pragma unroll
      for (int plane = 0; plane < 8; ++plane) {
        const bool on = plane == 0 ? (p >= 0) : (((mag >> (plane - 1)) & 1u) != 0u);
        const uint32_t piece = every_fourth_bit(__ballot(on));  // rows 16 (wid + rr NT / 64) .. + 15
        if (lane == 0) o.qc16[plane * (L / 16) + rr * (NT / 64) + wid] = (uint16_t)piece;
      }
    }
  }
  __syncthreads();
}

// The group sum of one row of P for the quad lane c that holds coordinates
// [32 c, 32 c + 32) of the row in pv (fp32, in coordinate order), with the
// group's queries in qs: the same fixed-order arithmetic as qpack_block (per
// head a sequential fp64 chain over the lane's 32 coordinates, the quad's
// four chains added as (c0 + c1) + (c2 + c3), the heads in ascending order).
// All four lanes of the quad must be active; each returns the row's value.
template <int G>
__device__ __forceinline__ double quad_row_sum(const float4 (&pv)[8], int c, const uint4 (*qs)[kHeadDim / 8]) {
  double xb = 0.0;
#pragma unroll
  for (int g0 = 0; g0 < G; g0 += 4) {
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float pf[8] = {pv[2 * j].x, pv[2 * j].y, pv[2 * j].z, pv[2 * j].w,
                           pv[2 * j + 1].x, pv[2 * j + 1].y, pv[2 * j + 1].z, pv[2 * j + 1].w};
      uint32_t w4[4][4];
#pragma unroll
      for (int hh = 0; hh < 4; ++hh) {
        const uint4 qq = qs[g0 + hh < G ? g0 + hh : g0][4 * c + j];
        w4[hh][0] = qq.x, w4[hh][1] = qq.y, w4[hh][2] = qq.z, w4[hh][3] = qq.w;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double d0 = (double)pf[2 * e], d1 = (double)pf[2 * e + 1];
#pragma unroll
        for (int hh = 0; hh < 4; ++hh) {
          acc[hh] = __builtin_fma(d0, (double)bf16_to_f32(w4[hh][e] & 0xFFFFu), acc[hh]);
          acc[hh] = __builtin_fma(d1, (double)bf16_to_f32(w4[hh][e] >> 16), acc[hh]);
        }
      }
    }
#pragma unroll
    for (int hh = 0; hh < 4; ++hh) {
      const double s01 = dadd(acc[hh], dpp_f64<kDppQuadXor1>(acc[hh]));
      const double a = dadd(s01, dpp_f64<kDppQuadXor2>(s01));
      if (g0 + hh < G) xb = (g0 + hh == 0) ? a : dadd(xb, a);
    }
  }
  return xb;
}

// ---------------------------------------------------------------------------
// 1. score -- one 512-thread workgroup per slice.
// The workgroup first packs its (b, h)'s query group (above).  Each thread
// then scores 32 keys with 16-byte non-temporal loads (a ring of kScanRing
// loads in flight) and keeps their distances in registers, two per
// register; the slice histogram lives in LDS.
// ---------------------------------------------------------------------------
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
constexpr int kScanRing = 4;  // 16-byte code loads in flight per thread

// The 16 bytes of codes starting at key n (4 / W keys) of a slice of cnt
// keys.  Keys at or past cnt read as zero words and are never loaded.
template <int W>
__device__ __forceinline__ u32x4_t load_code_group(const uint32_t* cb, int n, int cnt, bool vec_ok) {
  constexpr int KPL = 4 / W;
  if (vec_ok && n + KPL <= cnt)
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(cb + (int64_t)n * W));
  uint32_t t4[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int u = 0; u < KPL; ++u)
    if (n + u < cnt)
#pragma unroll
      for (int w = 0; w < W; ++w) t4[u * W + w] = cb[(int64_t)(n + u) * W + w];
  return u32x4_t{t4[0], t4[1], t4[2], t4[3]};
}

// weighted Hamming distance sum_j 2^j popc(M_j & (code ^ s)) of key u of a
// 16-byte group, by Horner's rule over the planes (most significant first:
// d = 2 d + popcounts of plane j), so that every popcount accumulates into d
// (one AND-XOR and one popcount per plane and word, one shift per plane)
template <int W>
__device__ __forceinline__ uint32_t code_distance(const u32x4_t cw, int u, const uint32_t (&M)[7][W],
                                                  const uint32_t (&sg)[W]) {
  uint32_t d = 0;
#pragma unroll
  for (int j = 6; j >= 0; --j) {
    d += d;
#pragma unroll
    for (int w = 0; w < W; ++w) d = (uint32_t)__popc(M[j][w] & (cw[u * W + w] ^ sg[w])) + d;
  }
  return d;
}

template <int L>
struct ScoreShared {
  static constexpr int W = L / 32;
  static constexpr int NB = dist_bins(L);
  static constexpr int NBP = (NB + 127) & ~127;  // histogram padded to whole coarse bins
  union U {
    uint32_t hist[NBP];
    QpackShared<L> qp;  // the query packing, before the histogram is cleared
  } u;
  QpackOut<L> qo;
  uint32_t coarse[kCoarseBins];
  uint32_t cc[kCoarseBins + 1];
  int cnt[kScoreThreads / 64];  // candidates per wavefront
  int kth, cmin, that;
};

// FULL: the slice holds kSlice keys and its codes are 16-byte aligned, so no
// per-key bounds tests are needed and every load is one 16-byte load
template <int L, bool FULL>
__device__ __forceinline__ void score_body(ScoreShared<L>& sh, int bh, int s, const uint16_t* __restrict__ q,
                                           const float* __restrict__ P, int64_t sP_b, int64_t sP_h, int G,
                                           uint32_t* __restrict__ qcode_ws, uint32_t* __restrict__ qcode_out,
                                           const uint32_t* __restrict__ codes, int64_t sC_b, int64_t sC_h, int Hkv,
                                           int N, int k, int nslices, uint32_t* __restrict__ cand,
                                           uint32_t* __restrict__ meta, uint32_t* __restrict__ hist_fine,
                                           uint32_t* __restrict__ hist_cc, uint32_t* __restrict__ win,
                                           int32_t* __restrict__ score_out) {
  constexpr int W = L / 32;
  constexpr int NB = ScoreShared<L>::NB;
  constexpr int NBP = ScoreShared<L>::NBP;
  constexpr int FS = fine_stride(L);
  constexpr int NT = kScoreThreads;
  constexpr int PER = kSlice / NT;  // keys per thread
  constexpr int KPL = 4 / W;        // keys per 16-byte load
  constexpr int NLD = PER / KPL;    // loads per thread
  constexpr int RD = kScanRing < NLD ? kScanRing : NLD;  // loads in flight per thread
  constexpr int NW = NT / 64;
  constexpr int KPW = kSlice / NW;  // keys per wavefront: a contiguous run
  constexpr int KSTEP = 64 * KPL;   // keys per load of the wavefront
  static_assert(NW <= 64, "wavefront offsets are scanned by one wavefront");

  const int b = bh / Hkv, h = bh % Hkv;
  const int n0 = s * kSlice;
  const int cnt = min(kSlice, N - n0);
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const uint32_t* cb = codes + b * sC_b + h * sC_h + (int64_t)n0 * W;
  // a head's codes are W-word aligned; 16-byte loads need a 16-byte aligned base
  const bool vec_ok = (reinterpret_cast<uintptr_t>(cb) & 15u) == 0;
  // key of load it, slot u of this lane: wavefront wid owns keys
  // [wid KPW, (wid + 1) KPW); one load of the wavefront covers KSTEP
  // consecutive keys, lane l reading keys l KPL .. l KPL + KPL - 1 of them
  auto key_of = [&](int it, int u) -> int { return wid * KPW + it * KSTEP + lane * KPL + u; };
  auto load_group = [&](int r) -> u32x4_t {
    const int n = key_of(r, 0);
    if constexpr (FULL)  // whole slice, 16-byte aligned: one load, 32-bit offset from a uniform base
      return __builtin_nontemporal_load(
          reinterpret_cast<const u32x4_t*>(reinterpret_cast<const char*>(cb) + (uint32_t)n * (4u * W)));
    else
      return load_code_group<W>(cb, n, cnt, vec_ok);
  };

  // the query planes of (b, h); they are uniform (scalar registers).  Slice
  // 0 also stores them (and sum |p|) for the attention kernel and the
  // caller.  The first code load of the ring is issued behind the P loads
  // and lands while the query is packed; the other RD - 1 follow the packing
  // (more loads in flight during it delay P for the workgroups dispatched
  // later on the CU, and the step gets slower).
  u32x4_t cw[RD];
  qpack_block<L, NT, kMaxGroup>(sh.u.qp, sh.qo, q + ((size_t)b * Hkv * G + (size_t)h * G) * kHeadDim,
                                P + b * sP_b + h * sP_h, G, [&]() { cw[0] = load_group(0); });
  BPC_STAMP(1, 5);
  const uint32_t* qcw = reinterpret_cast<const uint32_t*>(sh.qo.qc16);
  uint32_t sg[W], M[7][W];
  int T = 0;  // sum |p_i| = sum_j 2^j popcount(plane 1 + j)
#pragma unroll
  for (int w = 0; w < W; ++w) {
    sg[w] = __builtin_amdgcn_readfirstlane(qcw[w]);
#pragma unroll
    for (int j = 0; j < 7; ++j) {
      M[j][w] = __builtin_amdgcn_readfirstlane(qcw[(1 + j) * W + w]);
      T += __popc(M[j][w]) << j;
    }
  }
  // a ring of RD code loads per thread stays in flight: the load of group
  // it + RD is issued as soon as group it has been consumed
#pragma unroll
  for (int r = 1; r < RD; ++r) cw[r] = load_group(r);
  if (s == 0 && threadIdx.x <= 8 * W) {
    const uint32_t v = threadIdx.x < 8 * W ? qcw[threadIdx.x] : (uint32_t)T;
    qcode_ws[(size_t)bh * kQcodeStride + threadIdx.x] = v;
    if (qcode_out && threadIdx.x < 8 * W) qcode_out[(size_t)bh * 8 * W + threadIdx.x] = v;
  }
  // the packing's LDS area is dead: every thread has passed the barrier
  // that ends qpack_block
#pragma unroll
  for (int r = 0; r < NBP / NT; ++r) sh.u.hist[r * NT + threadIdx.x] = 0u;
  __syncthreads();

  // distances (< 2^14) packed two per register: key i = it * KPL + u is half i & 1 of dpk[i >> 1]
  uint32_t dpk[PER / 2];
#pragma unroll
  for (int it = 0; it < NLD; ++it) {
    const u32x4_t c = cw[it % RD];
    if (it + RD < NLD) cw[it % RD] = load_group(it + RD);
#pragma unroll
    for (int u = 0; u < KPL; ++u) {
      // a key past the slice's end gets the distance 0xFFFF, above every bin
      const bool valid = FULL || key_of(it, u) < cnt;
      const uint32_t d = valid ? code_distance<W>(c, u, M, sg) : 0xFFFFu;
      const int i = it * KPL + u;
      dpk[i >> 1] = (i & 1) ? (dpk[i >> 1] | (d << 16)) : d;
      // opaque once packed: later reads must unpack rather than keep d alive
      if (i & 1) __asm__ volatile("" : "+v"(dpk[i >> 1]));
      if (valid) atomicAdd(&sh.u.hist[d], 1u);
    }
  }
  __syncthreads();
  BPC_STAMP(1, 1);
  auto dist_of = [&](int it, int u) -> int {
    const int i = it * KPL + u;
    return (int)((dpk[i >> 1] >> ((i & 1) << 4)) & 0xFFFFu);
  };
  auto is_cand = [&](int it, int u, int kth) -> bool {
    return dist_of(it, u) <= kth;  // kth < 0xFFFF
  };

  // ---- the histogram in 1024 segments of 16 bins, eight per coarse bin
  // (consecutive lanes): coarse counts, and the fine bins rewritten in place
  // in prefix form, (count in [128 (t >> 7), t)) << 16 | count at t
#pragma unroll
  for (int rr = 0; rr < 1024 / NT; ++rr) {
    const int seg = rr * NT + threadIdx.x;
    const int cbin = seg >> 3, part = seg & 7;
    const int fb0 = (cbin << kCoarseShift) + part * 16;
    uint32_t cntv[16];
    if (fb0 < NBP) {
      const uint4* hv = reinterpret_cast<const uint4*>(sh.u.hist + fb0);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint4 x = hv[r];
        cntv[4 * r] = x.x, cntv[4 * r + 1] = x.y, cntv[4 * r + 2] = x.z, cntv[4 * r + 3] = x.w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 16; ++e) cntv[e] = 0u;
    }
    int local = 0;
#pragma unroll
    for (int e = 0; e < 16; ++e) local += (int)cntv[e];
    const int incl = group8_inclusive_sum(local);
    if (part == 7) sh.coarse[cbin] = (uint32_t)incl;
    if (fb0 < NBP) {
      uint32_t run = (uint32_t)(incl - local);
      uint4* hv = reinterpret_cast<uint4*>(sh.u.hist + fb0);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        uint32_t v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[e] = (run << 16) | cntv[4 * r + e];
          run += cntv[4 * r + e];
        }
        hv[r] = make_uint4(v[0], v[1], v[2], v[3]);
      }
    }
  }
  __syncthreads();

  BPC_STAMP(1, 2);
  // wave 0: coarse prefix, the lowest occupied coarse bin, and the coarse
  // bins holding the slice's k-th key and its m-th key, m = ceil(k cnt / N)
  // (the slice's share of the budget: its own estimate of the threshold)
  const int mloc = (int)(((int64_t)k * cnt + N - 1) / N);
  if (threadIdx.x < 64) {
    const uint32_t c0 = sh.coarse[2 * lane], c1 = sh.coarse[2 * lane + 1];
    const int x = wave_inclusive_sum((int)(c0 + c1));
    const int ex = x - (int)(c0 + c1);
    sh.cc[2 * lane] = (uint32_t)ex;
    sh.cc[2 * lane + 1] = (uint32_t)ex + c0;
    if (lane == 63) sh.cc[kCoarseBins] = (uint32_t)x;
    const unsigned long long m0 = __ballot(ex + (int)c0 >= k);
    const unsigned long long m1 = __ballot(x >= k);
    const int f0 = first_lane(m0), f1 = first_lane(m1);
    const int cs = min(f0 < 64 ? 2 * f0 : 1 << 30, f1 < 64 ? 2 * f1 + 1 : 1 << 30);
    const unsigned long long n0m = __ballot(ex + (int)c0 >= mloc);
    const unsigned long long n1m = __ballot(x >= mloc);
    const int h0 = first_lane(n0m), h1 = first_lane(n1m);
    const int cs2 = min(h0 < 64 ? 2 * h0 : 1 << 30, h1 < 64 ? 2 * h1 + 1 : 1 << 30);
    const unsigned long long z0 = __ballot(c0 != 0u), z1 = __ballot(c1 != 0u);
    const int g0 = first_lane(z0), g1 = first_lane(z1);
    // the first fine bin of coarse bin c where the count reaches `need`
    // (NB - 1 when c < 0, i.e. the slice holds fewer than k keys): lane l
    // tests bins l and l + 64 of c, whose prefix form adds the count below c
    static_assert(kCoarseShift == 7, "two fine bins of a coarse bin per lane");
    auto fine_first = [&](int c, int need) -> int {
      if (c < 0 || c >= kCoarseBins) return NB - 1;
      const int below = __builtin_amdgcn_readlane((c & 1) ? ex + (int)c0 : ex, c >> 1);
      const int t0 = (c << kCoarseShift) + lane, t1 = t0 + 64;
      const uint32_t v0 = (t0 < NBP) ? sh.u.hist[t0] : 0u, v1 = (t1 < NBP) ? sh.u.hist[t1] : 0u;
      const unsigned long long r0 = __ballot(below + (int)(v0 >> 16) + (int)(v0 & 0xFFFFu) >= need);
      const unsigned long long r1 = __ballot(below + (int)(v1 >> 16) + (int)(v1 & 0xFFFFu) >= need);
      return r0 ? (c << kCoarseShift) + first_lane(r0) : r1 ? (c << kCoarseShift) + 64 + first_lane(r1) : NB - 1;
    };
    const int kth_w = fine_first((cnt >= k) ? cs : -1, k);
    const int that_w = fine_first(cs2, mloc);  // mloc <= cnt: always found
    if (lane == 0) {
      sh.kth = kth_w;
      sh.that = that_w;
      sh.cmin = min(g0 < 64 ? 2 * g0 : kCoarseBins - 1, g1 < 64 ? 2 * g1 + 1 : kCoarseBins - 1);
    }
  }
  __syncthreads();
  const int kth = sh.kth;
  const int cmin = sh.cmin;
  // The window: kWinBins distances ending `up` above the slice's estimate
  // t = sh.that, with `up` about six standard deviations of that estimate
  // (sqrt(mloc) keys over the local density of keys per distance), and the
  // largest distance a candidate may have, cand_max = min(t + up, kth); the
  // one-round threshold is only accepted at or below every slice's cand_max.
  int wbase, cand_max;
  {
    auto cumd = [&](int t) -> int {  // keys with distance <= t
      if (t < 0) return 0;
      if (t >= NBP) return cnt;
      const uint32_t v = sh.u.hist[t];
      return (int)(sh.cc[t >> kCoarseShift] + (v >> 16) + (v & 0xFFFFu));
    };
    const int that = sh.that;
    const int dens17 = max(cumd(that + 8) - cumd(that - 9), 1);  // keys in 17 distances around t
    const int up = min(max((int)ceilf(6.0f * sqrtf((float)mloc) * 17.0f / (float)dens17), 4), kWinBins - 32);
    wbase = max(that + up - (kWinBins - 1), 0);
    cand_max = min(that + up, kth);
  }
  BPC_STAMP(1, 3);

  // ---- histograms for the threshold: coarse prefix (129 entries) and the
  // fine bins in [128 cmin, kth] (bins below are empty, bins above are never
  // needed), coalesced from LDS
  const size_t sl = (size_t)bh * nslices + s;
  if (threadIdx.x <= kCoarseBins) hist_cc[sl * kCoarseStride + threadIdx.x] = sh.cc[threadIdx.x];
  {
    uint32_t* hf = hist_fine + sl * FS;
    for (int t = (cmin << kCoarseShift) + threadIdx.x; t <= kth; t += NT) hf[t] = sh.u.hist[t];
  }
  // ---- window record: cumulative counts over [wbase, wbase + kWinBins) as
  // u16 pairs (the histogram is in prefix form over all of [0, NBP))
  {
    uint32_t* wr = win + sl * kWinRec;
    auto cum = [&](int t) -> uint32_t {  // keys with distance <= t
      if (t >= NBP) return (uint32_t)cnt;
      const uint32_t v = sh.u.hist[t];
      return sh.cc[t >> kCoarseShift] + (v >> 16) + (v & 0xFFFFu);
    };
    if (threadIdx.x < kWinBins / 2)
      wr[4 + threadIdx.x] = cum(wbase + 2 * threadIdx.x) | (cum(wbase + 2 * threadIdx.x + 1) << 16);
    else if (threadIdx.x == kWinBins / 2)
      *reinterpret_cast<uint4*>(wr) =
          make_uint4((uint32_t)wbase, (uint32_t)cand_max, wbase > 0 ? cum(wbase - 1) : 0u, (uint32_t)cnt);
  }

  // ---- candidates (dist <= cand_max) in key order, which is (wavefront, it,
  // lane, u): the wavefronts' counts are scanned once, then each wavefront
  // writes its candidates from a running offset
  {
    int c = 0;
#pragma unroll
    for (int it = 0; it < NLD; ++it)
#pragma unroll
      for (int u = 0; u < KPL; ++u) c += is_cand(it, u, cand_max) ? 1 : 0;
    c = wave_inclusive_sum(c);  // lane 63: the wavefront's count
    if (lane == 63) sh.cnt[wid] = c;
  }
  // the write pass re-derives its flags instead of keeping PER comparison masks
#pragma unroll
  for (int i = 0; i < PER / 2; ++i) __asm__ volatile("" : "+v"(dpk[i]));
  __syncthreads();
  int total;  // the slice's candidate count
  {
    // every wavefront scans the NW counts itself: its own offset and the total
    const int v = (lane < NW) ? sh.cnt[lane] : 0;
    const int x = wave_inclusive_sum(v);
    total = __builtin_amdgcn_readlane(x, 63);
    uint32_t* cs_out = cand + sl * kSlice;
    int base = __builtin_amdgcn_readlane(x - v, wid);  // uniform over the wavefront
#pragma unroll
    for (int it = 0; it < NLD; ++it) {
      int pos = base;
      bool f[KPL];
#pragma unroll
      for (int u = 0; u < KPL; ++u) {
        f[u] = is_cand(it, u, cand_max);
        const unsigned long long m = __ballot(f[u]);
        pos += (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        base += (int)__popcll(m);
      }
#pragma unroll
      for (int u = 0; u < KPL; ++u)
        if (f[u]) cs_out[pos++] = ((uint32_t)key_of(it, u) << 16) | (uint32_t)dist_of(it, u);
    }
  }
  if (threadIdx.x == 0) *reinterpret_cast<uint4*>(meta + sl * 4) = make_uint4(kth, cmin, total, cand_max);
  if (score_out) {  // debug output
    int32_t* so = score_out + (size_t)bh * N + n0;
    int kb = wid * KPW + lane * KPL;  // opaque: no per-key offsets are kept from the scoring loop
    __asm__ volatile("" : "+v"(kb));
#pragma unroll
    for (int it = 0; it < NLD; ++it)
#pragma unroll
      for (int u = 0; u < KPL; ++u) {
        const int n = kb + it * KSTEP + u;
        if (n < cnt) so[n] = T - 2 * dist_of(it, u);
      }
  }
}

// four 512-thread workgroups per CU (8 wavefronts per SIMD) at L <= 64: the
// whole grid of a 128K-key batch is resident at once.  FULL = true handles
// the slices that hold kSlice keys with 16-byte aligned codes, FULL = false
// the others (a ragged last slice, or codes with strides that are not a
// multiple of four words); each launch skips the other kind, and the second
// is only launched when such slices exist.
template <int L, bool FULL>
__global__ __launch_bounds__(kScoreThreads) __attribute__((amdgpu_waves_per_eu(L <= 64 ? 8 : 4))) void score_kernel(
    const uint16_t* __restrict__ q, const float* __restrict__ P, int64_t sP_b, int64_t sP_h, int G,
    uint32_t* __restrict__ qcode_ws, uint32_t* __restrict__ qcode_out, const uint32_t* __restrict__ codes,
    int64_t sC_b, int64_t sC_h, int BH,
    int Hkv, int N, int k, int nslices, uint32_t* __restrict__ cand, uint32_t* __restrict__ meta,
    uint32_t* __restrict__ hist_fine, uint32_t* __restrict__ hist_cc, uint32_t* __restrict__ win,
    int32_t* __restrict__ score_out) {
  __shared__ ScoreShared<L> sh;
  int bh, s;
  slice_tile(blockIdx.x, BH, nslices, bh, s);
  const int64_t c0 = (int64_t)(bh / Hkv) * sC_b + (int64_t)(bh % Hkv) * sC_h + (int64_t)s * kSlice * (L / 32);
  const bool full = (s + 1) * kSlice <= N && (reinterpret_cast<uintptr_t>(codes + c0) & 15u) == 0;
  if (full != FULL) return;
  BPC_STAMP(1, 0);
  score_body<L, FULL>(sh, bh, s, q, P, sP_b, sP_h, G, qcode_ws, qcode_out, codes, sC_b, sC_h, Hkv, N, k, nslices, cand, meta, hist_fine, hist_cc,
                      win, score_out);
  BPC_STAMP(1, 4);
}

// ---------------------------------------------------------------------------
// 2. attend -- one 256-thread workgroup per slice.
//  a. Threshold: the coarse prefixes of every slice of (b, h) give the coarse
//     bin c* of the k-th smallest distance, their fine bins in c* give T*
//     and the number of keys at T* still to take; keys below T* and ties at
//     T* in the earlier slices give this slice's quota of ties (ties go to
//     the lowest indices, i.e. slice by slice) and its output offset.  The
//     histograms of up to kPlanCache slices are kept in LDS, which saves a
//     round of loads.
//  b. Selection: the slice's candidates, kCandBatch at a time, are kept if
//     their distance is below T* or at T* within the quota; the kept keys
//     (ascending) go to the LDS row list and to idx_out.
//  c. Attention: each wavefront runs independently over rows of the list,
//     16 per pass; every K and V load of a pass is issued before the first
//     is consumed.  The logits of the pass's 16 rows and the group's query
//     heads are one 16 x 16 x 128 product on the matrix cores (rows x heads,
//     heads padded to 16), in base 2 (sm_scale * log2 e); they reach the
//     lanes holding the V rows through LDS.  Sixteen lanes share a V row
//     (lane l16 holds dims [8 l16, 8 l16 + 8)), and the wavefront carries
//     its own running (max, sum, weighted V).  The four wavefronts are
//     combined once, into one partial per query head.
// ---------------------------------------------------------------------------
typedef short bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// D += A B for one 16 x 16 x 16 bf16 tile (fp32 accumulation).  Lane i
// supplies A[i % 16][4 (i / 16) + j] and B[4 (i / 16) + j][i % 16] (j = 0..3,
// two bf16 per 32-bit word, low half first) and holds D[4 (i / 16) + j][i % 16].
__device__ __forceinline__ f32x4_t mfma16(uint32_t a0, uint32_t a1, uint32_t b0, uint32_t b1, f32x4_t d) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(bf16x4_t, make_uint2(a0, a1)),
                                                   __builtin_bit_cast(bf16x4_t, make_uint2(b0, b1)), d, 0, 0, 0);
}

__device__ __forceinline__ void unpack8(const uint4 v, float (&f)[8]) {
  f[0] = bf16_to_f32(v.x & 0xFFFFu), f[1] = bf16_to_f32(v.x >> 16);
  f[2] = bf16_to_f32(v.y & 0xFFFFu), f[3] = bf16_to_f32(v.y >> 16);
  f[4] = bf16_to_f32(v.z & 0xFFFFu), f[5] = bf16_to_f32(v.z >> 16);
  f[6] = bf16_to_f32(v.w & 0xFFFFu), f[7] = bf16_to_f32(v.w >> 16);
}

constexpr int kAttnWaves = kAttnThreads / 64;
constexpr int kAttnRows = 16;                // rows per wavefront per pass (one 16-row tile)
constexpr int kPlanCache = 16;               // slices whose histograms are kept in LDS
constexpr int kRoundBatch = 8;               // histogram loads per thread issued together
constexpr int kRowCache = 2048;              // selected rows kept in LDS (more go through global memory)

template <int G>
struct AttendShared {
  // two-round threshold (any slice count)
  struct Plan {
    int part[2][kCoarseBins], part2[2][kCoarseBins];
    int gp[kCoarseBins];
    uint32_t cc[kPlanCache][kCoarseBins + 1];      // coarse prefix of each slice
    uint32_t fine[kPlanCache][1 << kCoarseShift];  // fine bins of c* of each slice
    int kth[kPlanCache], cmin[kPlanCache];
  };
  union alignas(16) U {
    Plan plan;
    uint32_t win[kWinSlices][kWinRec];  // one-round threshold: the window records of the slices
    int rows[kRowCache];                // the slice's selected keys, ascending
    float o[kAttnWaves][G][kHeadDim];   // per-wavefront weighted V
  } u;
  float st[kAttnWaves][G][2];  // per wavefront (max, sum)
  alignas(16) float pl[kAttnWaves][G][16];  // per wavefront: the logits of a pass, handed between lanes
  uint4 q[G][kHeadDim / 8];     // the group's queries, bf16
  int wave_tot[2][kAttnWaves];  // block scans, double-buffered
  int first[2];
  int red[2][kAttnWaves];
  uint32_t sel[kSlice / 32];  // the safeguard: bitmap of the slice's keys the hash selection took
};

// An empty instruction that reads and rewrites x: loads feeding it are all
// waited for here, together.
__device__ __forceinline__ void pin_regs(uint4& x) {
  __asm__ volatile("" : "+v"(x.x), "+v"(x.y), "+v"(x.z), "+v"(x.w));
}

// One pass of a wavefront over nrows (1..kAttnRows) rows; lane (r, c) =
// (lane / 16, lane % 16) holds the key index of row c in rk and those of
// rows 4 r .. 4 r + 3 in rv (key 0 for a row at or past nrows: it exists in
// every head, and its logit is masked); pl is the wavefront's [G][16] LDS
// area for the logits.  Updates the wavefront's running maximum Mx and sum
// Ls (uniform over the wavefront) and this lane's weighted-V partials o.
//
// Logits: lane (r, c) = (lane / 16, lane % 16) loads dims [32 kb + 8 r, +8)
// of K row c (kb = 0..3) and, as the second operand, the same dims of query
// head c (zero for c >= G); each 16-byte load feeds two tiles (dims +0..3
// and +4..7), so eight tiles cover the 128 dims.  The result, D[row][head],
// lands in lane (r, head) for rows 4 r .. 4 r + 3.  V: lane (r, c) loads
// dims [8 c, 8 c + 8) of rows 4 r .. 4 r + 3, which are exactly the rows
// whose logits the lanes (r, head < G) of its own group hold.
// The pieces of one pass: the K loads, the V loads, the logits (from K) and
// the softmax update with the weighted V (from V).  attend_pass runs them in
// order; a pipelined caller issues the next pass's loads between them.  The
// rows are read once: non-temporal loads keep them from displacing what the
// caches hold for the other workgroups (measured: 4.5 us of the decode step
// at batch 16 x 8 x 131072 against plain loads).
__device__ __forceinline__ void attend_load_k(uint32_t rk, const char* Kh, uint32_t kstride, uint4 (&kv)[4]) {
  const int r4 = (threadIdx.x & 63) >> 4;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    const u32x4_t x =
        __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(Kh + (rk * kstride + 64u * kb + 16u * r4)));
    kv[kb] = make_uint4(x[0], x[1], x[2], x[3]);
  }
}
__device__ __forceinline__ void attend_load_v(const uint32_t (&rv)[4], const char* Vh, uint32_t vstride,
                                              uint4 (&vv)[4]) {
  const int c16 = threadIdx.x & 15;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const u32x4_t x = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(Vh + (rv[t] * vstride + 16u * c16)));
    vv[t] = make_uint4(x[0], x[1], x[2], x[3]);
  }
}

template <int G>
__device__ __forceinline__ void attend_logits(const uint4 (&kv)[4], int nrows, const uint4 (*qs)[kHeadDim / 8],
                                              float scale_log2, float& mx, float& ls, float& f, float (&x)[4]);
template <int G>
__device__ __forceinline__ void attend_pv(const uint4 (&vv)[4], float (*pl)[16], float f, float (&o)[G][8]);

// mx, ls: the running (max, sum) of query head lane % 16 (lanes below G)
template <int G>
__device__ __forceinline__ void attend_pass(uint32_t rk, const uint32_t (&rv)[4], int nrows,
                                            const uint4 (*qs)[kHeadDim / 8], float (*pl)[16], const char* Kh,
                                            uint32_t kstride, const char* Vh, uint32_t vstride, float scale_log2,
                                            float& mx, float& ls, float (&o)[G][8]) {
  uint4 kv[4], vv[4];
  attend_load_k(rk, Kh, kstride, kv);
  attend_load_v(rv, Vh, vstride, vv);
  float f, pr[4];
  attend_logits<G>(kv, nrows, qs, scale_log2, mx, ls, f, pr);
  if ((threadIdx.x & 15) < G)
    *reinterpret_cast<float4*>(&pl[threadIdx.x & 15][4 * ((threadIdx.x & 63) >> 4)]) = make_float4(pr[0], pr[1], pr[2], pr[3]);
  attend_pv<G>(vv, pl, f, o);
}

// Logits of the pass's rows (from their K) and the running softmax update,
// computed in the lanes that hold them: lane (r, g) = (lane / 16, lane % 16),
// g < G, has the logits of rows 4 r .. 4 r + 3 for query head g and keeps head
// g's running maximum mx and sum ls (the same in its four row groups).  The
// pass's probabilities come back in x (zero in lanes g >= G), the rescale
// factor of earlier passes in f.  The arithmetic is that of a
// wavefront-uniform update: the maximum over the four row groups, then
// exp2(logit - max), the group sums added as ((r0 + r1) + (r2 + r3)).
template <int G>
__device__ __forceinline__ void attend_logits(const uint4 (&kv)[4], int nrows, const uint4 (*qs)[kHeadDim / 8],
                                              float scale_log2, float& mx, float& ls, float& f, float (&x)[4]) {
  static_assert(G <= 16, "the query heads of a group fill at most the 16 columns of a tile");
  const int lane = threadIdx.x & 63;
  const int c16 = lane & 15, r4 = lane >> 4;
  // logits on the matrix cores
  int qi = c16;
  __asm__ volatile("" : "+v"(qi));  // the query is re-read from LDS each pass, not held in registers
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    const uint4 qv = qi < G ? qs[qi][4 * kb + r4] : make_uint4(0u, 0u, 0u, 0u);
    acc = mfma16(kv[kb].x, kv[kb].y, qv.x, qv.y, acc);
    acc = mfma16(kv[kb].z, kv[kb].w, qv.z, qv.w, acc);
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) x[j] = 4 * r4 + j < nrows ? acc[j] * scale_log2 : -INFINITY;
  // the pass's maximum over the 16 rows: the lane's four, then across the row groups
  float m = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
  {
    const auto p16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(m), __float_as_uint(m), false, false);
    m = fmaxf(__uint_as_float(p16[0]), __uint_as_float(p16[1]));
    const auto p32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
    m = fmaxf(__uint_as_float(p32[0]), __uint_as_float(p32[1]));
  }
  const float mnew = fmaxf(mx, m);
  // rescale what earlier passes accumulated (mx = -inf before the first: factor 0)
  f = (mx == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mx - mnew);
  float ps = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    x[j] = __builtin_amdgcn_exp2f(x[j] - mnew);  // a masked row: exp2(-inf) = 0
    ps += x[j];
  }
  {
    const auto p16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(ps), __float_as_uint(ps), false, false);
    const float y = __uint_as_float(p16[0]) + __uint_as_float(p16[1]);
    const auto p32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
    ps = __uint_as_float(p32[0]) + __uint_as_float(p32[1]);
  }
  ls = ls * f + ps;
  mx = mnew;
  if (c16 >= G)
#pragma unroll
    for (int j = 0; j < 4; ++j) x[j] = 0.f;
}

// The weighted V of the pass whose probabilities are in pl, after scaling
// what earlier passes accumulated by each head's factor f (lane g holds
// head g's).
template <int G>
__device__ __forceinline__ void attend_pv(const uint4 (&vv)[4], float (*pl)[16], float f, float (&o)[G][8]) {
  const int lane = threadIdx.x & 63;
  const int r4 = lane >> 4;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const float fg = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), g));
    if (fg != 1.f)  // a product with 1 changes nothing
#pragma unroll
      for (int e = 0; e < 8; ++e) o[g][e] *= fg;
  }
  // LDS operations of one wavefront complete in order: the reads below see
  // the writes above; this only keeps the compiler from moving them across
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  float lg[G][4];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const float4 x = *reinterpret_cast<const float4*>(&pl[g][4 * r4]);
    lg[g][0] = x.x, lg[g][1] = x.y, lg[g][2] = x.z, lg[g][3] = x.w;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();  // the next pass rewrites pl only after these reads
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  // weighted V of the lane's rows
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    float vf[8];
    unpack8(vv[t], vf);
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < 8; ++e) o[g][e] = fmaf(lg[g][t], vf[e], o[g][e]);
  }
}

// The weighted V on the matrix cores.  D[head][dim] += P[head][row] V[row][dim]
// for the pass's 16 rows is one 16 x 16 x 16 bf16 tile per 16 dims (heads
// padded to 16 rows of D).  The A operand is the probabilities, which lane
// (r, g) already holds for rows 4 r .. 4 r + 3 of head g, split into a bf16
// high part and a bf16 low part (p - high), so the products keep about 16
// significant bits of p and are accumulated in fp32 (two tiles per 16 dims).
// The B operand wants, in lane (r, c), the four rows of dim 16 T + c: each
// row group (16 lanes, rows 4 r .. 4 r + 3) stores its four V rows dim-major
// ([dim][4 rows] bf16, 8 bytes per dim) in the wavefront's LDS area vt, and
// every lane reads one 8-byte entry per tile.  Lane (r, c) accumulates
// D[4 r + j][16 T + c] in acc[T][j].
constexpr int kVtGroupBytes = kHeadDim * 8 + 16;  // one row group's block (padded: the groups start in other banks)
constexpr int kVtWaveBytes = 4 * kVtGroupBytes;

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t bf16x2_bits(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

template <int G>
__device__ __forceinline__ void attend_pv_mfma(const uint4 (&vv)[4], const float (&pr)[4], float f, char* vt,
                                               f32x4_t (&acc)[8]) {
  const int lane = threadIdx.x & 63;
  const int c16 = lane & 15, r4 = lane >> 4;
  // rescale what earlier passes accumulated: D row j of this lane is head 4 r + j
  if (__any(c16 < G && f != 1.f)) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float fj = G <= 4 ? __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), j))
                              : __shfl(f, 4 * r4 + j);
#pragma unroll
      for (int T = 0; T < 8; ++T) acc[T][j] *= fj;
    }
  }
  // the row group's four rows, dim-major: dims 8 c + 2 m and 8 c + 2 m + 1 are
  // the halves of word m of each row
  char* grp = vt + r4 * kVtGroupBytes;
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const uint32_t w0 = (&vv[0].x)[m], w1 = (&vv[1].x)[m], w2 = (&vv[2].x)[m], w3 = (&vv[3].x)[m];
    uint4 d;
    d.x = __builtin_amdgcn_perm(w1, w0, 0x05040100u);  // dim 2m: rows 0, 1
    d.y = __builtin_amdgcn_perm(w3, w2, 0x05040100u);  //         rows 2, 3
    d.z = __builtin_amdgcn_perm(w1, w0, 0x07060302u);  // dim 2m + 1: rows 0, 1
    d.w = __builtin_amdgcn_perm(w3, w2, 0x07060302u);  //             rows 2, 3
    *reinterpret_cast<uint4*>(grp + (8 * c16 + 2 * m) * 8) = d;
  }
  // the probabilities as bf16 high and low parts
  const uint32_t h01 = bf16x2_bits(pr[0], pr[1]), h23 = bf16x2_bits(pr[2], pr[3]);
  const uint32_t l01 = bf16x2_bits(pr[0] - __uint_as_float(h01 << 16), pr[1] - __uint_as_float(h01 & 0xFFFF0000u));
  const uint32_t l23 = bf16x2_bits(pr[2] - __uint_as_float(h23 << 16), pr[3] - __uint_as_float(h23 & 0xFFFF0000u));
  // LDS operations of one wavefront complete in order; the fences only keep
  // the compiler from moving the reads above the writes
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
  for (int T = 0; T < 8; ++T) {
    const uint2 bv = *reinterpret_cast<const uint2*>(grp + (16 * T + c16) * 8);
    acc[T] = mfma16(h01, h23, bv.x, bv.y, acc[T]);
    acc[T] = mfma16(l01, l23, bv.x, bv.y, acc[T]);
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();  // the next pass rewrites vt only after these reads
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One pass with the weighted V on the matrix cores (see attend_pass).
template <int G>
__device__ __forceinline__ void attend_pass_mfma(uint32_t rk, const uint32_t (&rv)[4], int nrows,
                                                 const uint4 (*qs)[kHeadDim / 8], char* vt, const char* Kh,
                                                 uint32_t kstride, const char* Vh, uint32_t vstride, float scale_log2,
                                                 float& mx, float& ls, f32x4_t (&acc)[8]) {
  uint4 kv[4], vv[4];
  attend_load_k(rk, Kh, kstride, kv);
  attend_load_v(rv, Vh, vstride, vv);
  float f, pr[4];
  attend_logits<G>(kv, nrows, qs, scale_log2, mx, ls, f, pr);
  attend_pv_mfma<G>(vv, pr, f, vt, acc);
}

// The running (max, sum) of each head as wavefront-uniform values, from the
// lanes that hold them.
template <int G>
__device__ __forceinline__ void lane_stats(float mx, float ls, float (&Mx)[G], float (&Ls)[G]) {
#pragma unroll
  for (int g = 0; g < G; ++g) {
    Mx[g] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mx), g));
    Ls[g] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ls), g));
  }
}

// Data one workgroup publishes for others of the same launch: agent-scope
// atomic stores and loads (coherent across the XCDs' L2 caches without a
// write-back of the L2), ordered by stores_complete() before the arrival.
__device__ __forceinline__ void pub_store(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t pub_load(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// every store this thread has issued is complete before anything after it
__device__ __forceinline__ void stores_complete() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void pub_store64(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t pub_load64(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The workgroup's partial for each query head g: each wavefront reduces its
// weighted V over its four row groups; the wavefronts are combined under
// their common maximum into pb[g] = (max, sum, o[128]) (base-2 logits).
// o_s and st_s are LDS arrays; the caller ensures o_s is free to write.
template <int G, bool PUBLISH>
__device__ __forceinline__ void combine_partial(const float (&o_s)[kAttnWaves][G][kHeadDim],
                                                const float (&st_s)[kAttnWaves][G][2], float* __restrict__ pb);

template <int G, bool PUBLISH = false>  // PUBLISH: agent-scope atomic stores (read by the merging workgroup)
__device__ __forceinline__ void write_partial(float (&o_s)[kAttnWaves][G][kHeadDim], float (&st_s)[kAttnWaves][G][2],
                                              const float (&Mx)[G], const float (&Ls)[G], float (&o)[G][8],
                                              float* __restrict__ pb) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, l16 = lane & 15;
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      // x[l] + x[l ^ 16], then + the same over l ^ 32: with both operands
      // equal, the two results of a permlane swap sum to exactly that
      const uint32_t x = __float_as_uint(o[g][e]);
      const auto p16 = __builtin_amdgcn_permlane16_swap(x, x, false, false);
      const uint32_t y = __float_as_uint(__uint_as_float(p16[0]) + __uint_as_float(p16[1]));
      const auto p32 = __builtin_amdgcn_permlane32_swap(y, y, false, false);
      o[g][e] = __uint_as_float(p32[0]) + __uint_as_float(p32[1]);
    }
  if (lane < 16) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < 8; ++e) o_s[wid][g][8 * l16 + e] = o[g][e];
  }
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) st_s[wid][g][0] = Mx[g], st_s[wid][g][1] = Ls[g];
  }
  __syncthreads();
  combine_partial<G, PUBLISH>(o_s, st_s, pb);
}

// write_partial for weighted V held as the matrix-core tiles of
// attend_pv_mfma (already summed over the wavefront's rows).
template <int G, bool PUBLISH = false>
__device__ __forceinline__ void write_partial_tiles(float (&o_s)[kAttnWaves][G][kHeadDim],
                                                    float (&st_s)[kAttnWaves][G][2], const float (&Mx)[G],
                                                    const float (&Ls)[G], const f32x4_t (&acc)[8],
                                                    float* __restrict__ pb) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int c16 = lane & 15, r4 = lane >> 4;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if (4 * r4 + j < G)
#pragma unroll
      for (int T = 0; T < 8; ++T) o_s[wid][4 * r4 + j][16 * T + c16] = acc[T][j];
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) st_s[wid][g][0] = Mx[g], st_s[wid][g][1] = Ls[g];
  }
  __syncthreads();
  combine_partial<G, PUBLISH>(o_s, st_s, pb);
}

// The wavefronts' partials, in o_s and st_s, combined under their common
// maximum into pb[g] = (max, sum, o[128]).
template <int G, bool PUBLISH>
__device__ __forceinline__ void combine_partial(const float (&o_s)[kAttnWaves][G][kHeadDim],
                                                const float (&st_s)[kAttnWaves][G][2], float* __restrict__ pb) {
  for (int e = threadIdx.x; e < G * (kHeadDim + 2); e += kAttnThreads) {
    const int g = e / (kHeadDim + 2), d = e % (kHeadDim + 2);
    float m = -INFINITY;
#pragma unroll
    for (int w = 0; w < kAttnWaves; ++w) m = fmaxf(m, st_s[w][g][0]);
    float acc = 0.f;
    if (d == 0) {
      acc = m;
    } else {
#pragma unroll
      for (int w = 0; w < kAttnWaves; ++w) {
        const float mw = st_s[w][g][0];
        const float f = (mw == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mw - m);
        acc = fmaf(d == 1 ? st_s[w][g][1] : o_s[w][g][d - 2], f, acc);
      }
    }
    if constexpr (PUBLISH)
      pub_store(reinterpret_cast<uint32_t*>(pb) + e, __float_as_uint(acc));
    else
      pb[e] = acc;
  }
}

template <int G>
__global__ __launch_bounds__(kAttnThreads) __attribute__((amdgpu_waves_per_eu(G <= 4 ? 4 : 1))) void attend_kernel(
    int N, int k, int L, int BH, int Hkv, int nslices, int win_ok, const uint32_t* __restrict__ cand,
    const uint32_t* __restrict__ meta, const uint32_t* __restrict__ hist_fine, const uint32_t* __restrict__ hist_cc,
    const uint32_t* __restrict__ win, const uint32_t* __restrict__ codes, int64_t sC_b, int64_t sC_h,
    const uint32_t* __restrict__ qcode, int32_t* __restrict__ idx_out, const int32_t* __restrict__ serr, int64_t sS_b,
    int64_t sS_h, int m, int32_t* __restrict__ added_out, const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ K, int64_t sK_b, int64_t sK_h, int64_t sK_n, const uint16_t* __restrict__ V,
    int64_t sV_b, int64_t sV_h, int64_t sV_n, float scale_log2, float* __restrict__ part) {
  constexpr int PER = kCandBatch / kAttnThreads;  // candidates per thread per batch
  __shared__ AttendShared<G> sh;
  typename AttendShared<G>::Plan& pl = sh.u.plan;
  int bh, s;
  slice_tile(blockIdx.x, BH, nslices, bh, s);
  const int b = bh / Hkv, h = bh % Hkv;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, l16 = lane & 15;
  const size_t sl = (size_t)bh * nslices + s;
  const uint32_t* cs = cand + sl * kSlice;
  const int n0 = s * kSlice;
  const int NB = dist_bins(L), FS = fine_stride(L);
  const bool cached = nslices <= kPlanCache;
  const uint32_t* ccb = hist_cc + (size_t)bh * nslices * kCoarseStride;
  const uint32_t* hfb = hist_fine + (size_t)bh * nslices * FS;
  const uint32_t* mtb = meta + (size_t)bh * nslices * 4;
  BPC_STAMP(2, 0);

  // ---- a. threshold: T*, the number `take` of this slice's keys at T* that
  // are selected, this slice's offset `off` in the (b, h) index list and the
  // number `kept` of keys it selects
  int tstar = 0, take = 0, off = 0, kept = 0, ncand = 0;
  bool planned = false;
  uint32_t cv[PER];  // this thread's current batch of (key << 16 | distance) entries
  auto load_cand = [&](int base) {  // a batch of the slice's candidate list
    const uint4 x = *reinterpret_cast<const uint4*>(cs + base + threadIdx.x * PER);
    cv[0] = x.x, cv[1] = x.y, cv[2] = x.z, cv[3] = x.w;
  };
  static_assert(PER == 4, "one 16-byte load of candidates per thread and batch");
  auto load_queries = [&]() {  // the group's queries, staged in LDS
    if (threadIdx.x < G * kHeadDim / 8) {
      const uint4* qb = reinterpret_cast<const uint4*>(q + ((size_t)b * Hkv * G + (size_t)h * G) * kHeadDim);
      sh.q[threadIdx.x / (kHeadDim / 8)][threadIdx.x % (kHeadDim / 8)] = qb[threadIdx.x];
    }
  };
  if (win_ok) {
    // One round: the window records of every slice of (b, h) (at most
    // kWinSlices).  Every window covers [lo - 1, hi] with lo = max_s base_s
    // and hi = min_s cand_max_s <= min_s (base_s + kWinBins - 1).  When
    // S(lo - 1) < k <= S(hi), with S(t) = sum_s cum_s(t), T* = lo +
    // #{t in [lo, hi] : S(t) < k} <= hi, so every slice's candidate list
    // holds all of its keys with distance <= T*; otherwise the two-round
    // path runs.
    constexpr int RV = (kWinSlices * kWinRec / 4 + kAttnThreads - 1) / kAttnThreads;
    const int nv = nslices * (kWinRec / 4);
    const uint4* wsrc = reinterpret_cast<const uint4*>(win + (size_t)bh * nslices * kWinRec);
    // every load of the round is unconditional (indices clamped), so that all
    // of them are in flight before the first wait
    uint4 wv[RV];
#pragma unroll
    for (int r = 0; r < RV; ++r) wv[r] = wsrc[min((int)threadIdx.x + r * kAttnThreads, nv - 1)];
    const uint4 mym = *reinterpret_cast<const uint4*>(mtb + s * 4);
    load_cand(0);
    uint4 qv = reinterpret_cast<const uint4*>(q + ((size_t)b * Hkv * G + (size_t)h * G) * kHeadDim)[min(
        (int)threadIdx.x, G * kHeadDim / 8 - 1)];
    // the values are taken here, so the compiler cannot sink each load into
    // the conditional store that uses it (which would wait on them one by one)
#pragma unroll
    for (int r = 0; r < RV; ++r) pin_regs(wv[r]);
    pin_regs(qv);
    if (threadIdx.x < G * kHeadDim / 8) sh.q[threadIdx.x / (kHeadDim / 8)][threadIdx.x % (kHeadDim / 8)] = qv;
    BPC_STAMP(2, 1);
    uint4* wdst = reinterpret_cast<uint4*>(&sh.u.win[0][0]);
#pragma unroll
    for (int r = 0; r < RV; ++r)
      if ((int)threadIdx.x + r * kAttnThreads < nv) wdst[threadIdx.x + r * kAttnThreads] = wv[r];
    ncand = min((int)mym.z, kSlice);
    __syncthreads();
    auto cum = [&](int u, int t) -> int {  // base_u - 1 <= t < base_u + kWinBins
      const int j = t - (int)sh.u.win[u][0];
      const uint32_t w = sh.u.win[u][4 + (max(j, 0) >> 1)];
      return (j < 0) ? (int)sh.u.win[u][2] : (int)((j & 1) ? (w >> 16) : (w & 0xFFFFu));
    };
    // lane u holds slice u's window (base, cand_max); lo and hi for every lane
    const int lo = wave_reduce_maxmin<true>(lane < nslices ? (int)sh.u.win[lane][0] : 0);
    const int hi = wave_reduce_maxmin<false>(lane < nslices ? (int)sh.u.win[lane][1] : (1 << 30));
    // thread i evaluates S(t) at t = lo - 1 + i (hi - lo + 2 <= kWinBins + 1 <= kAttnThreads values); the
    // counts of t in [lo, hi] with S(t) < k and the failed checks go through ballots
    bool below = false, badt = false;
    const int t = lo - 1 + (int)threadIdx.x;
    if (lo <= hi && t <= hi) {
      int St = 0;
#pragma unroll 8
      for (int u = 0; u < nslices; ++u) St += cum(u, t);
      if (t == lo - 1)
        badt = St >= k;
      else
        below = St < k;
      if (t == hi && St < k) badt = true;
    }
    const unsigned long long mbelow = __ballot(below), mbad = __ballot(badt);
    if (lane == 0) sh.red[0][wid] = (int)__popcll(mbelow), sh.red[1][wid] = mbad != 0ull;
    __syncthreads();
    BPC_STAMP(2, 2);
    int cntlow = 0, bad = lo > hi;
#pragma unroll
    for (int w = 0; w < kAttnWaves; ++w) cntlow += sh.red[0][w], bad |= sh.red[1][w];
    if (!bad) {
      tstar = lo + cntlow;
      // every wavefront derives its slice's plan from the windows, lane u for
      // slice u: keys below T* and ties at T*, and their prefix sums over the
      // slices; ties go to the lowest indices, i.e. the slices before s take
      // min(need, their ties) of the `need` ties
      int bu = 0, tu = 0;
      if (lane < nslices) {
        bu = cum(lane, tstar - 1);
        tu = cum(lane, tstar) - bu;
      }
      const int bi = wave_inclusive_sum(bu), ti = wave_inclusive_sum(tu);
      const int below_all = __builtin_amdgcn_readlane(bi, 63);
      const int below_before = __builtin_amdgcn_readlane(bi - bu, s), ties_before = __builtin_amdgcn_readlane(ti - tu, s);
      const int bs = __builtin_amdgcn_readlane(bu, s), ts = __builtin_amdgcn_readlane(tu, s);
      const int need = k - below_all;  // keys at T* to take, over all slices
      take = max(0, min(ts, need - ties_before));
      off = below_before + min(need, ties_before);
      kept = bs + take;
      planned = true;
    }
    __syncthreads();  // the window area is reused below
  }
  if (!planned) {
    // Two rounds.  Round 1: GP(c + 1) = keys of all slices with coarse bin
    // <= c.  Each round's loads are issued together: kRoundBatch slices per
    // thread at a time, the slice index clamped so every load is
    // unconditional, and entries past the last slice dropped after the load.
    {
      const int c = threadIdx.x & (kCoarseBins - 1), grp = threadIdx.x >> 7;
      int acc = 0;
      for (int u0 = grp; u0 < nslices; u0 += 2 * kRoundBatch) {
        uint32_t v[kRoundBatch];
#pragma unroll
        for (int j = 0; j < kRoundBatch; ++j)
          v[j] = ccb[(size_t)min(u0 + 2 * j, nslices - 1) * kCoarseStride + c + 1];
#pragma unroll
        for (int j = 0; j < kRoundBatch; ++j) {
          const int u = u0 + 2 * j;
          if (u < nslices) {
            acc += (int)v[j];
            if (cached) pl.cc[u][c + 1] = v[j];
          }
        }
      }
      pl.part[grp][c] = acc;
      if (cached && threadIdx.x < nslices) {
        const uint4 m = *reinterpret_cast<const uint4*>(mtb + threadIdx.x * 4);
        pl.cc[threadIdx.x][0] = 0u;
        pl.kth[threadIdx.x] = min((int)m.x, NB - 1);
        pl.cmin[threadIdx.x] = min((int)m.y, kCoarseBins - 1);
      }
    }
    if (!win_ok) load_queries();  // else already staged
    __syncthreads();
    if (threadIdx.x < kCoarseBins) {
      const int acc = pl.part[0][threadIdx.x] + pl.part[1][threadIdx.x];
      pl.gp[threadIdx.x] = acc;
      const unsigned long long m = __ballot(acc >= k);
      if (lane == 0) sh.first[wid] = m ? first_lane(m) + 64 * wid : (1 << 30);
    }
    __syncthreads();
    const int cstar = min(min(sh.first[0], sh.first[1]), kCoarseBins - 1);
    const int below_c = (cstar > 0) ? pl.gp[cstar - 1] : 0;  // keys with coarse bin < c*
    __syncthreads();
    // Round 2: the fine bins of c*, summed over slices (bins a slice did not
    // write are empty below its cmin and never needed above its kth)
    {
      const int j = threadIdx.x & ((1 << kCoarseShift) - 1), grp = threadIdx.x >> 7;
      const int t = (cstar << kCoarseShift) + j;
      const int tc = min(t, NB - 1);
      int exc = 0, inc = 0;
      for (int u0 = grp; u0 < nslices; u0 += 2 * kRoundBatch) {
        int kthu[kRoundBatch], cminu[kRoundBatch];
        uint32_t v[kRoundBatch];
#pragma unroll
        for (int i = 0; i < kRoundBatch; ++i) {
          const int u = min(u0 + 2 * i, nslices - 1);
          if (cached) {
            kthu[i] = pl.kth[u], cminu[i] = pl.cmin[u];
          } else {
            const uint2 m = *reinterpret_cast<const uint2*>(mtb + u * 4);
            kthu[i] = (int)m.x, cminu[i] = (int)m.y;
          }
          v[i] = hfb[(size_t)u * FS + tc];  // a bin the slice did not write is dropped below
        }
#pragma unroll
        for (int i = 0; i < kRoundBatch; ++i) {
          const int u = u0 + 2 * i;
          if (u < nslices) {
            const uint32_t x = (t < NB && t >= (cminu[i] << kCoarseShift) && t <= kthu[i]) ? v[i] : 0u;
            if (cached) pl.fine[u][j] = x;
            exc += (int)(x >> 16);
            inc += (int)(x >> 16) + (int)(x & 0xFFFFu);
          }
        }
      }
      pl.part[grp][j] = exc;
      pl.part2[grp][j] = inc;
    }
    __syncthreads();
    if (threadIdx.x < (1 << kCoarseShift)) {
      const int exc = pl.part[0][threadIdx.x] + pl.part[1][threadIdx.x];
      const int inc = pl.part2[0][threadIdx.x] + pl.part2[1][threadIdx.x];
      const int t = (cstar << kCoarseShift) + threadIdx.x;
      const unsigned long long m = __ballot(t < NB && below_c + inc >= k);
      if (lane == 0) sh.first[wid] = m ? first_lane(m) + 64 * wid : (1 << 30);
      pl.gp[threadIdx.x] = exc;
    }
    __syncthreads();
    const int jt = min(min(sh.first[0], sh.first[1]), (1 << kCoarseShift) - 1);
    tstar = min((cstar << kCoarseShift) + jt, NB - 1);
    const int need = k - (below_c + pl.gp[jt]);  // keys at T* to take, over all slices
    // Round 3: keys below T* and ties at T* of the slices before this one
    // (and this slice's own ties).  The slices before s take min(need, their
    // ties) of the ties; this slice takes what is left, up to its own.
    auto slice_at_tstar = [&](int u, int& below, int& tie) {
      uint32_t v;
      int ccv;
      if (cached) {
        v = pl.fine[u][jt];
        ccv = (int)pl.cc[u][cstar];
      } else {
        const int cminu = (int)mtb[u * 4 + 1];
        v = (tstar >= (cminu << kCoarseShift)) ? hfb[(size_t)u * FS + tstar] : 0u;
        ccv = (int)ccb[(size_t)u * kCoarseStride + cstar];
      }
      below = ccv + (int)(v >> 16);
      tie = (int)(v & 0xFFFFu);
    };
    int bl = 0, ti = 0;
    for (int u = threadIdx.x; u < s; u += kAttnThreads) {
      int bu, tu;
      slice_at_tstar(u, bu, tu);
      bl += bu, ti += tu;
    }
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      bl += __shfl_xor(bl, o, 64);
      ti += __shfl_xor(ti, o, 64);
    }
    if (lane == 0) sh.red[0][wid] = bl, sh.red[1][wid] = ti;
    int my_below, my_tie;
    slice_at_tstar(s, my_below, my_tie);
    __syncthreads();
    int below_before = 0, ties_before = 0;
#pragma unroll
    for (int w = 0; w < kAttnWaves; ++w) below_before += sh.red[0][w], ties_before += sh.red[1][w];
    take = max(0, min(my_tie, need - ties_before));
    off = below_before + min(need, ties_before);
    kept = my_below + take;
    __syncthreads();  // the plan area is reused below
  }
  kept = min(kept, k - off);
  BPC_STAMP(2, 3);

  // ---- b. selection: the kept entries, in ascending key order, go to the
  // slice's row list (in LDS when it holds them and the safeguard keys,
  // else over the slice's own candidate area: a kept entry's rank never
  // exceeds its position there, and the safeguard keys are appended after
  // every candidate has been read) and, when the caller asks for them, to
  // [off, off + kept) of the (b, h) index list.  In the one-round path the
  // entries are the slice's candidate list (it holds every key with distance
  // <= T* since T* <= hi <= cand_max_s); otherwise the slice's codes are
  // scored again.
  const bool rows_lds = kept + m <= kRowCache;
  int32_t* grows = reinterpret_cast<int32_t*>(const_cast<uint32_t*>(cs));
  int32_t* xrows = idx_out ? idx_out + (size_t)bh * k + off : nullptr;
  if (m > 0)
    for (int i = threadIdx.x; i < kSlice / 32; i += kAttnThreads) sh.sel[i] = 0u;  // ordered by the scan's barriers
  const int nent = planned ? ncand : min(kSlice, N - n0);
  const int W = L / 32;
  uint32_t sg[4] = {0u, 0u, 0u, 0u}, M[7][4] = {};
  const uint32_t* cb = codes + b * sC_b + h * sC_h + (int64_t)n0 * W;
  if (!planned) {
    const uint32_t* qc = qcode + (size_t)bh * kQcodeStride;
#pragma unroll
    for (int w = 0; w < 4; ++w)
      if (w < W) {
        sg[w] = qc[w];
#pragma unroll
        for (int j = 0; j < 7; ++j) M[j][w] = qc[(1 + j) * W + w];
      }
  }
  auto rescore = [&](int base) {  // entries of keys base + PER t + e, scored from their codes
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int key = base + (int)threadIdx.x * PER + e;
      uint32_t d = 0;
      if (key < nent) {
#pragma unroll
        for (int w = 0; w < 4; ++w)
          if (w < W) {
            const uint32_t x = cb[(int64_t)key * W + w] ^ sg[w];
#pragma unroll
            for (int j = 0; j < 7; ++j) d += (uint32_t)__popc(M[j][w] & x) << j;
          }
      }
      cv[e] = ((uint32_t)key << 16) | d;
    }
  };
  int nkept = 0, tie_seen = 0;  // kept keys and ties at T* in earlier batches
  int sbuf = 0;                 // block scans alternate their LDS totals
  for (int base = 0; base < nent; base += kCandBatch) {
    if (!planned)
      rescore(base);
    else if (base > 0)
      load_cand(base);
    // distances of this thread's entries; entries past the count never match
    const int nvalid = nent - base - (int)threadIdx.x * PER;
    int nb = 0, nt = 0;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int d = (e < nvalid) ? (int)(cv[e] & 0xFFFFu) : (1 << 30);
      nb += d < tstar;
      nt += d == tstar;
    }
    int tot;
    // one scan of packed (ties << 16 | below): at most kCandBatch of each per batch
    const int pre = block_exclusive_scan_bits<kAttnThreads, 0x70007u>((nt << 16) | nb, sh.wave_tot, sbuf, tot);
    sbuf ^= 1;
    int tie_rank = tie_seen + (pre >> 16);
    int rank = nkept + (pre & 0xFFFF) + max(0, min(tie_rank, take) - min(tie_seen, take));
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int d = (e < nvalid) ? (int)(cv[e] & 0xFFFFu) : (1 << 30);
      bool keep = d < tstar;
      if (d == tstar) {
        keep = tie_rank < take;
        ++tie_rank;
      }
      if (keep && rank < kept) {
        const int kin = (int)(cv[e] >> 16);
        if (rows_lds)
          sh.u.rows[rank] = n0 + kin;
        else
          grows[rank] = n0 + kin;
        if (xrows) xrows[rank] = n0 + kin;
        if (m > 0) atomicOr(&sh.sel[kin >> 5], 1u << (kin & 31));
      }
      rank += keep;
    }
    nkept += (tot & 0xFFFF) + max(0, min(tie_seen + (tot >> 16), take) - min(tie_seen, take));
    tie_seen += tot >> 16;
  }
  __syncthreads();  // the list is complete and visible to the whole workgroup

  // ---- error-aware safeguard: the keys of S_err in this slice that the hash
  // selection did not take are appended to the row list (in S_err order,
  // which is ascending); added_out marks them
  if (m > 0) {
    const int32_t* se = serr + b * sS_b + h * sS_h;
    const int cnt = min(kSlice, N - n0);
    int extra = 0;
    for (int base = 0; base < m; base += 4 * kAttnThreads) {
      int key[4], add[4], na = 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = base + 4 * (int)threadIdx.x + u;
        key[u] = (j < m) ? se[j] : -1;
        const int kin = key[u] - n0;
        const bool here = key[u] >= n0 && kin < cnt;
        add[u] = here && !((sh.sel[kin >> 5] >> (kin & 31)) & 1u);
        // an entry outside [0, N) lies in no slice: slice 0 marks it as not added
        const bool outside = j < m && (key[u] < 0 || key[u] >= N);
        if (added_out && (here || (outside && s == 0))) added_out[(size_t)bh * m + j] = add[u];
        na += add[u];
      }
      int tot;
      int pos = kept + extra + block_exclusive_scan_bits<kAttnThreads, 0x7u>(na, sh.wave_tot, sbuf, tot);
      sbuf ^= 1;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (add[u]) {
          if (rows_lds)
            sh.u.rows[pos] = key[u];  // pos < kept + m <= kRowCache
          else if (pos < kSlice)      // (repeated S_err entries could overrun the area)
            grows[pos] = key[u];
          ++pos;
        }
      extra += tot;
    }
    kept = min(kept + extra, rows_lds ? kRowCache : kSlice);
    __syncthreads();
  }
  BPC_STAMP(2, 4);

  // ---- c. attention: wavefront wid takes rows [16 (wid + 4 i), 16 (wid + 4 i) + 16)
  const char* Kh = reinterpret_cast<const char*>(K + b * sK_b + h * sK_h);
  const char* Vh = reinterpret_cast<const char*>(V + b * sV_b + h * sV_h);
  const uint32_t kstride = (uint32_t)sK_n * 2u, vstride = (uint32_t)sV_n * 2u;
  float mx = -INFINITY, ls = 0.f;  // running (max, sum) of query head lane % 16 (lanes below G)
  float o[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
#pragma unroll
    for (int e = 0; e < 8; ++e) o[g][e] = 0.f;
  }
  // lane (r, c) reads the key indices of row c and rows 4 r .. 4 r + 3 of
  // the pass from the row list (entries at or past kept are masked; the
  // list's area holds r0 + 15 since r0 is a multiple of 16 below kept)
  auto pass_rows = [&](const int32_t* rl, int r0, int nr, uint32_t& rk, uint32_t (&rv)[4]) {
    const int c16 = lane & 15, r4 = lane >> 4;
    const int kc = rl[r0 + c16];
    const int4 v4 = *reinterpret_cast<const int4*>(rl + r0 + 4 * r4);
    rk = c16 < nr ? (uint32_t)kc : 0u;
    rv[0] = 4 * r4 + 0 < nr ? (uint32_t)v4.x : 0u;
    rv[1] = 4 * r4 + 1 < nr ? (uint32_t)v4.y : 0u;
    rv[2] = 4 * r4 + 2 < nr ? (uint32_t)v4.z : 0u;
    rv[3] = 4 * r4 + 3 < nr ? (uint32_t)v4.w : 0u;
  };
  if (rows_lds) {
    for (int r0 = wid * kAttnRows; r0 < kept; r0 += kAttnWaves * kAttnRows) {
      const int nr = min(kAttnRows, kept - r0);
      uint32_t rk, rv[4];
      pass_rows(sh.u.rows, r0, nr, rk, rv);
      attend_pass<G>(rk, rv, nr, sh.q, sh.pl[wid], Kh, kstride, Vh, vstride, scale_log2, mx, ls, o);
    }
  } else {
    for (int r0 = wid * kAttnRows; r0 < kept; r0 += kAttnWaves * kAttnRows) {
      const int nr = min(kAttnRows, kept - r0);
      uint32_t rk, rv[4];
      pass_rows(grows, r0, nr, rk, rv);
      attend_pass<G>(rk, rv, nr, sh.q, sh.pl[wid], Kh, kstride, Vh, vstride, scale_log2, mx, ls, o);
    }
  }
  BPC_STAMP(2, 5);
  BPC_NOTE(2, 12, kept);
  BPC_NOTE(2, 13, ncand);
  BPC_NOTE(2, 14, planned);
  __syncthreads();  // the row list is read to the end before its area holds o

  float Mx[G], Ls[G];
  lane_stats<G>(mx, ls, Mx, Ls);
  write_partial<G>(sh.u.o, sh.st, Mx, Ls, o, part + sl * G * (kHeadDim + 2));
  BPC_STAMP(2, 6);
}

// ---------------------------------------------------------------------------
// Dense decode attention over all N keys: the comparison point the paper's
// efficiency numbers are quoted against (full attention at decode), not part
// of the method.  One 256-thread workgroup per chunk of kSlice consecutive
// keys of a (b, h); each wavefront takes runs of 16 consecutive rows with the
// same row pass as the sparse kernel; the partials go through merge_kernel.
// ---------------------------------------------------------------------------
template <int G>
struct DenseShared {
  float o[kAttnWaves][G][kHeadDim];
  float st[kAttnWaves][G][2];
  alignas(16) float pl[kAttnWaves][G][16];
  uint4 q[G][kHeadDim / 8];
};

template <int G>
__global__ __launch_bounds__(kAttnThreads) __attribute__((amdgpu_waves_per_eu(G <= 4 ? 4 : 1))) void dense_kernel(
    int N, int Hkv, int nchunks, const uint16_t* __restrict__ q, const uint16_t* __restrict__ K, int64_t sK_b,
    int64_t sK_h, int64_t sK_n, const uint16_t* __restrict__ V, int64_t sV_b, int64_t sV_h, int64_t sV_n,
    float scale_log2, float* __restrict__ part) {
  __shared__ DenseShared<G> sh;
  const int bh = blockIdx.x / nchunks, s = blockIdx.x % nchunks;
  const int b = bh / Hkv, h = bh % Hkv;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  if (threadIdx.x < G * kHeadDim / 8) {
    const uint4* qb = reinterpret_cast<const uint4*>(q + ((size_t)b * Hkv * G + (size_t)h * G) * kHeadDim);
    sh.q[threadIdx.x / (kHeadDim / 8)][threadIdx.x % (kHeadDim / 8)] = qb[threadIdx.x];
  }
  __syncthreads();
  const int n0 = s * kSlice, cnt = min(kSlice, N - n0);
  const char* Kh = reinterpret_cast<const char*>(K + b * sK_b + h * sK_h);
  const char* Vh = reinterpret_cast<const char*>(V + b * sV_b + h * sV_h);
  const uint32_t kstride = (uint32_t)sK_n * 2u, vstride = (uint32_t)sV_n * 2u;
  float mx = -INFINITY, ls = 0.f;  // running (max, sum) of query head lane % 16 (lanes below G)
  float o[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
#pragma unroll
    for (int e = 0; e < 8; ++e) o[g][e] = 0.f;
  }
  for (int r0 = wid * kAttnRows; r0 < cnt; r0 += kAttnWaves * kAttnRows) {
    const int nr = min(kAttnRows, cnt - r0);
    const int c16 = lane & 15, r4 = lane >> 4;
    const uint32_t rk = c16 < nr ? (uint32_t)(n0 + r0 + c16) : 0u;
    uint32_t rv[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) rv[t] = 4 * r4 + t < nr ? (uint32_t)(n0 + r0 + 4 * r4 + t) : 0u;
    attend_pass<G>(rk, rv, nr, sh.q, sh.pl[wid], Kh, kstride, Vh, vstride, scale_log2, mx, ls, o);
  }
  float Mx[G], Ls[G];
  lane_stats<G>(mx, ls, Mx, Ls);
  write_partial<G>(sh.o, sh.st, Mx, Ls, o, part + (size_t)blockIdx.x * G * (kHeadDim + 2));
}

// ---------------------------------------------------------------------------
// 3. merge -- one workgroup per (b, query head): log-sum-exp combination of
// the slice partials (a slice that selected nothing has max -inf, sum 0).
// A separate launch, rather than a last-workgroup merge inside the attention
// kernel: there every workgroup would have to wait for its partial stores
// before counting itself in, which lengthens each of them.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kHeadDim) void merge_kernel(int Hkv, int G, int nchunks, const float* __restrict__ part,
                                                         float* __restrict__ out) {
  constexpr int MB = 8;  // partials per batch: all of a batch's loads are issued before the first is used
  const int bq = blockIdx.x;  // b * Hq + query head
  const int Hq = Hkv * G;
  const int b = bq / Hq, jq = bq % Hq;
  const int h = jq / G, g = jq % G;
  const size_t bh = (size_t)b * Hkv + h;
  const size_t cstride = (size_t)G * (kHeadDim + 2);
  const float* pg = part + bh * nchunks * cstride + (size_t)g * (kHeadDim + 2);
  const int d = threadIdx.x;
  BPC_STAMP(3, 0);
  // one pass with a running maximum: each thread reads every partial's
  // (max, sum) and its own coordinate of the weighted V
  float M = -INFINITY, lsum = 0.f, acc = 0.f;
  for (int t0 = 0; t0 < nchunks; t0 += MB) {
    float mt[MB], lt[MB], ot[MB];
#pragma unroll
    for (int u = 0; u < MB; ++u) {
      const float* pc = pg + (size_t)min(t0 + u, nchunks - 1) * cstride;
      mt[u] = pc[0], lt[u] = pc[1], ot[u] = pc[2 + d];
    }
    float mb = -INFINITY;
#pragma unroll
    for (int u = 0; u < MB; ++u) {
      if (t0 + u >= nchunks) mt[u] = -INFINITY;  // past the last partial: dropped
      mb = fmaxf(mb, mt[u]);
    }
    const float Mn = fmaxf(M, mb);
    if (Mn == -INFINITY) continue;  // no partial with a key so far
    const float f = (M == -INFINITY) ? 0.f : exp2f(M - Mn);
    lsum *= f, acc *= f;
#pragma unroll
    for (int u = 0; u < MB; ++u) {
      const float w = (mt[u] == -INFINITY) ? 0.f : exp2f(mt[u] - Mn);
      lsum = fmaf(lt[u], w, lsum);
      acc = fmaf(ot[u], w, acc);
    }
    M = Mn;
  }
  out[(size_t)bq * kHeadDim + d] = acc / lsum;
  BPC_STAMP(3, 1);
}

// ===========================================================================
// Fused decode step: the whole step in one launch, one 256-thread workgroup
// per slice, every workgroup of the grid resident at once (the host checks
// the occupancy).  A workgroup
//  1. packs its (b, h)'s query group and scores its slice (64 keys per lane,
//     distances kept in registers, an LDS histogram);
//  2. publishes its window record, its histogram summary and its coarse
//     prefix, then waits until every slice of (b, h) has published;
//  3. derives T*, its tie quota and its output offset from the records (the
//     one-round window rule of the attention kernel above; else the exact
//     two rounds, the second publishing the fine bins of the coarse bin c*);
//  4. selects its kept keys straight from its registers, in key order,
//     gathers their K/V rows and accumulates its softmax partial;
//  5. publishes the partial; the last workgroup of (b, h) to do so merges the
//     partials of every slice into the output and returns the (b, h)'s
//     arrival counters to zero for the next call.
// Handoffs between workgroups use agent-scope atomic stores and loads for
// the published data, a wait for the stores' completion, and a relaxed
// agent-scope counter: the published data are visible to any workgroup once
// the counter shows their writer's arrival, with no L2 write-back.  The only
// wait is bounded; it is never reached when the grid is resident, and a
// workgroup that reaches it keeps no rows.
// ===========================================================================
constexpr int kFusedThreads = 256;
constexpr int kFusedWaves = kFusedThreads / 64;
constexpr int kFusedRing = 8;              // 16-byte code loads in flight per thread
constexpr unsigned kSpinLimit = 1u << 22;  // bounded wait on the arrival counter
// published per slice: the window record, (kth, cmin, count, window end), the
// coarse prefix (129 counts) and, in the exact two-round path, the counts of
// the 128 fine bins of c*
constexpr int kPubMeta = kWinRec;
constexpr int kPubCoarse = kPubMeta + 4;
constexpr int kPubFine = kPubCoarse + kCoarseStride;
constexpr int kPubStride = kPubFine + (1 << kCoarseShift);
static_assert(kPubStride == kFusedPubWords, "published record size");


// Sum over the nslices slices of (b, h) of f(published word of slice u),
// kBatch loads per thread in flight before the first is used.
constexpr int kBatch = 8;
template <class Addr, class F>
__device__ __forceinline__ int sum_published(int nslices, Addr addr, F f) {
  int acc = 0;
  for (int u0 = 0; u0 < nslices; u0 += kBatch) {
    uint32_t v[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) v[j] = pub_load(addr(min(u0 + j, nslices - 1)));
#pragma unroll
    for (int j = 0; j < kBatch; ++j) acc += (u0 + j < nslices) ? f(v[j]) : 0;
  }
  return acc;
}
// Copy nv published words, word e from src(e), to dst[e] in LDS; R loads per
// thread are in flight before the first is used.
template <int R, class T, class Src>
__device__ __forceinline__ void copy_published(T* dst, int nv, Src src) {
  for (int e0 = 0; e0 < nv; e0 += R * kFusedThreads) {
    T v[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int e = e0 + (int)threadIdx.x + r * kFusedThreads;
      v[r] = (e < nv) ? T(sizeof(T) == 8 ? pub_load64(reinterpret_cast<const uint64_t*>(src(e)))
                                         : pub_load(reinterpret_cast<const uint32_t*>(src(e))))
                      : T(0);
    }
    // the values are taken here, so that the compiler cannot sink each load
    // into the conditional store that uses it (and wait on them one by one)
#pragma unroll
    for (int r = 0; r < R; ++r) __asm__ volatile("" : "+v"(v[r]));
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int e = e0 + (int)threadIdx.x + r * kFusedThreads;
      if (e < nv) dst[e] = v[r];
    }
  }
}

template <int L, int G>
struct FusedShared {
  static constexpr int NB = dist_bins(L);
  static constexpr int NBP = (NB + 127) & ~127;
  struct Attn {
    uint32_t win[kWinSlices][kWinRec];  // window records of the (b, h)'s slices (one-round threshold)
    int rows[kRowCache];                // the candidates (key << 16 | distance), then over them the
                                        // first kRowCache selected keys in rank order
    uint32_t sel[kSlice / 32];          // the safeguard: bitmap of the slice's keys the hash selection took
  };
  union alignas(16) U {
    uint32_t hist[NBP];
    QpackShared<L, G> qp;
    Attn at;
    float o[kFusedWaves][G][kHeadDim];
  } u;
  QpackOut<L> qo;
  uint32_t coarse[kCoarseBins];
  uint32_t cc[kCoarseBins + 1];
  uint32_t fine[1 << kCoarseShift];  // counts of the fine bins of c* (two-round path)
  int gsum[2][kCoarseBins];          // two-round path: sums over slices
  int wcnt[kFusedWaves][2];          // per wavefront: keys below T*, ties at T*
  int kth, cmin, that, flag;
  int red[2][kFusedWaves];
  int wave_tot[2][kFusedWaves];
  float st[kFusedWaves][G][2];
  alignas(16) float pl[kFusedWaves][G][16];
  uint4 q[G][kHeadDim / 8];
};

// waves per SIMD the kernel is built for: four 256-thread workgroups per CU
// (the 1024-slice grid of a batch of 16 x 8 heads x 128K keys resident) where
// LDS allows it; L = 128 holds 64 KB of histogram, so two
static_assert(kVtWaveBytes * kFusedWaves <= (int)sizeof(uint32_t) * kWinSlices * kWinRec,
              "the weighted-V transposes of the wavefronts fit in the window area");

template <int L, int G>
constexpr int fused_waves() { return L == 128 ? 2 : G <= 4 ? 4 : G == 8 ? 3 : 1; }

template <int L, int G, int SL>
__global__ __launch_bounds__(kFusedThreads) __attribute__((amdgpu_waves_per_eu(fused_waves<L, G>()))) void fused_decode_kernel(
    const uint16_t* __restrict__ q, const float* __restrict__ P, int64_t sP_b, int64_t sP_h,
    const uint32_t* __restrict__ codes, int64_t sC_b, int64_t sC_h, const uint16_t* __restrict__ K, int64_t sK_b,
    int64_t sK_h, int64_t sK_n, const uint16_t* __restrict__ V, int64_t sV_b, int64_t sV_h, int64_t sV_n, int BH,
    int Hkv, int N, int k, int nslices, float scale_log2, uint32_t* __restrict__ sync, uint32_t* __restrict__ pub,
    float* __restrict__ part, int32_t* __restrict__ rows, float* __restrict__ out, int32_t* __restrict__ idx_out,
    int32_t* __restrict__ score_out, uint32_t* __restrict__ qcode_out, const int32_t* __restrict__ serr, int64_t sS_b,
    int64_t sS_h, int m, int32_t* __restrict__ added_out, int ncu) {
  constexpr int W = L / 32;
  constexpr int NT = kFusedThreads;
  constexpr int NW = kFusedWaves;
  constexpr int NB = FusedShared<L, G>::NB;
  constexpr int NBP = FusedShared<L, G>::NBP;
  constexpr int PER = SL / NT;          // keys per thread
  constexpr int KPL = 4 / W;             // keys per 16-byte load
  constexpr int NLD = PER / KPL;         // loads per thread
  constexpr int RD = kFusedRing < NLD ? kFusedRing : NLD;
  constexpr int KPW = SL / NW;          // keys per wavefront: a contiguous run
  constexpr int KSTEP = 64 * KPL;        // keys per load of the wavefront
  __shared__ FusedShared<L, G> sh;

  int bh, s;
  slice_tile(blockIdx.x, BH, nslices, bh, s);
  const int b = bh / Hkv, h = bh % Hkv;
  const int n0 = s * SL;
  const int cnt = min(SL, N - n0);
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const size_t sl = (size_t)bh * nslices + s;
  uint32_t* my_pub = pub + sl * kPubStride;
  const uint32_t* bh_pub = pub + (size_t)bh * nslices * kPubStride;
  uint32_t* bh_sync = sync + (size_t)bh * kFusedSyncWords;
  BPC_STAMP(1, 0);

  // ---- 1. query packing and scoring -----------------------------------
  const uint32_t* cb = codes + b * sC_b + h * sC_h + (int64_t)n0 * W;
  const bool full = cnt == SL && (reinterpret_cast<uintptr_t>(cb) & 15u) == 0;
  auto key_of = [&](int it, int u) -> int { return wid * KPW + it * KSTEP + lane * KPL + u; };
  auto load_group = [&](int r) -> u32x4_t {
    const int n = key_of(r, 0);
    if (full)
      return __builtin_nontemporal_load(
          reinterpret_cast<const u32x4_t*>(reinterpret_cast<const char*>(cb) + (uint32_t)n * (4u * W)));
    return load_code_group<W>(cb, n, cnt, (reinterpret_cast<uintptr_t>(cb) & 15u) == 0);
  };
  u32x4_t cw[RD];
  const uint16_t* qg = q + ((size_t)b * Hkv * G + (size_t)h * G) * kHeadDim;
  const float* Pbh = P + b * sP_b + h * sP_h;
  // the (b, h)'s shared query rows (an expression, not a value kept live)
  auto xq_of = [&]() {
    return reinterpret_cast<uint64_t*>(sync + (size_t)kFusedMaxBH * kFusedSyncWords) + (size_t)bh * kFusedMaxL;
  };
  if (nslices == 1) {
    qpack_block<L, NT, G>(sh.u.qp, sh.qo, qg, Pbh, G, [&]() { cw[0] = load_group(0); });
  } else {
    // The slices of (b, h) share the projection: slice s computes rows
    // [s R, s R + R) of the group sum (R = ceil(L / nslices)) and publishes
    // them (bit-complemented, so that a published row is never zero); every
    // slice then collects all L rows and quantises them itself.  The rows go
    // back to zero when the step's merge ends.
    const int R = (L + nslices - 1) / nslices;
    const int r0 = s * R, nr = max(0, min(R, L - r0));
    const int i = threadIdx.x >> 2, c = threadIdx.x & 3;  // quad i: row r0 + i
    if (threadIdx.x < G * (kHeadDim / 8))
      sh.q[threadIdx.x / (kHeadDim / 8)][threadIdx.x % (kHeadDim / 8)] = reinterpret_cast<const uint4*>(qg)[threadIdx.x];
    float4 pv[8];
    if (i < nr) {
      const float4* pr = reinterpret_cast<const float4*>(Pbh + (size_t)(r0 + i) * kHeadDim + 32 * c);
#pragma unroll
      for (int j = 0; j < 8; ++j) pv[j] = pr[j];
    }
    cw[0] = load_group(0);
    __syncthreads();  // the queries
    BPC_STAMP(1, 6);
    if (i < nr) {
      const double x = quad_row_sum<G>(pv, c, sh.q);
      if (c == 0) pub_store64(xq_of() + r0 + i, ~(uint64_t)__double_as_longlong(x));
    }
    if (wid == 0) {
      // every row published (rows at or past L count as present)
      uint64_t v0 = lane < L ? 0u : 1u, v1 = lane + 64 < L ? 0u : 1u;
      unsigned it = 0;
      for (;;) {
        if (v0 == 0u) v0 = pub_load64(xq_of() + lane);
        if (v1 == 0u) v1 = pub_load64(xq_of() + 64 + lane);
        if (__all(v0 != 0u && v1 != 0u) || ++it >= kSpinLimit) break;
        __builtin_amdgcn_s_sleep(2);
      }
      // a row still missing after the bounded wait counts as zero
      const double x0 = (lane < L && v0 != 0u) ? __longlong_as_double((long long)~v0) : 0.0;
      const double x1 = (lane + 64 < L && v1 != 0u) ? __longlong_as_double((long long)~v1) : 0.0;
      double m = fmax(fabs(x0), fabs(x1));
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) {
        const int lo = __shfl_xor(__double2loint(m), off), hi = __shfl_xor(__double2hiint(m), off);
        m = fmax(m, __hiloint2double(hi, lo));
      }
      const int p0 = (m > 0.0) ? (int)round(dmul(x0, 127.0) / m) : 0;
      const int p1 = (m > 0.0) ? (int)round(dmul(x1, 127.0) / m) : 0;
      uint32_t* qw = reinterpret_cast<uint32_t*>(sh.qo.qc16);
#pragma unroll
      for (int plane = 0; plane < 8; ++plane) {
        const bool on0 = plane == 0 ? (p0 >= 0) : (((uint32_t)abs(p0) >> (plane - 1)) & 1u) != 0u;
        const bool on1 = plane == 0 ? (p1 >= 0) : (((uint32_t)abs(p1) >> (plane - 1)) & 1u) != 0u;
        const unsigned long long m0 = __ballot(on0 && lane < L), m1 = __ballot(on1 && lane + 64 < L);
        if (lane == 0) {
          qw[plane * W] = (uint32_t)m0;
          if (W > 1) qw[plane * W + 1] = (uint32_t)(m0 >> 32);
          if (W > 2) qw[plane * W + 2] = (uint32_t)m1, qw[plane * W + 3] = (uint32_t)(m1 >> 32);
        }
      }
    }
    __syncthreads();
  }
  BPC_STAMP(1, 1);
  const uint32_t* qcw = reinterpret_cast<const uint32_t*>(sh.qo.qc16);
  uint32_t sg[W], M[7][W];
  int T = 0;  // sum |p_i|
#pragma unroll
  for (int w = 0; w < W; ++w) {
    sg[w] = __builtin_amdgcn_readfirstlane(qcw[w]);
#pragma unroll
    for (int j = 0; j < 7; ++j) {
      M[j][w] = __builtin_amdgcn_readfirstlane(qcw[(1 + j) * W + w]);
      T += __popc(M[j][w]) << j;
    }
  }
  // Scoring runs at a wave priority that grows with the workgroup's dispatch
  // round (its age rank on the CU: ids [r ncu, (r + 1) ncu) are dispatched in
  // round r).  The memory system serves the older workgroups of a CU first,
  // so the youngest finish scoring last and their selection and attention
  // end the step; raising their priority evens the rounds out (70.2 against
  // 68.5 us per step at batch 16 x 131072 keys).
  switch (min(3, (int)blockIdx.x / ncu)) {
    case 1: __builtin_amdgcn_s_setprio(1); break;
    case 2: __builtin_amdgcn_s_setprio(2); break;
    case 3: __builtin_amdgcn_s_setprio(3); break;
    default: break;
  }
#pragma unroll
  for (int r = 1; r < RD; ++r) cw[r] = load_group(r);
  if (s == 0 && qcode_out && threadIdx.x < 8 * W) qcode_out[(size_t)bh * 8 * W + threadIdx.x] = qcw[threadIdx.x];
  for (int r = threadIdx.x; r < NBP; r += NT) sh.u.hist[r] = 0u;
  __syncthreads();
  // distances (< 2^14) two per register: key i = it * KPL + u is half i & 1 of dpk[i >> 1]
  uint32_t dpk[PER / 2];
  if (full) {  // every key of the slice present, every load one 16-byte load: no per-key tests
#pragma unroll
    for (int it = 0; it < NLD; ++it) {
      const u32x4_t c = cw[it % RD];
      if (it + RD < NLD)
        cw[it % RD] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(
            reinterpret_cast<const char*>(cb) + (uint32_t)key_of(it + RD, 0) * (4u * W)));
#pragma unroll
      for (int u = 0; u < KPL; ++u) {
        const uint32_t d = code_distance<W>(c, u, M, sg);
        const int i = it * KPL + u;
        dpk[i >> 1] = (i & 1) ? (dpk[i >> 1] | (d << 16)) : d;
        if (i & 1) __asm__ volatile("" : "+v"(dpk[i >> 1]));
        atomicAdd(&sh.u.hist[d], 1u);
      }
    }
  } else {
#pragma unroll
    for (int it = 0; it < NLD; ++it) {
      const u32x4_t c = cw[it % RD];
      if (it + RD < NLD) cw[it % RD] = load_group(it + RD);
#pragma unroll
      for (int u = 0; u < KPL; ++u) {
        const bool valid = key_of(it, u) < cnt;
        const uint32_t d = valid ? code_distance<W>(c, u, M, sg) : 0xFFFFu;
        const int i = it * KPL + u;
        dpk[i >> 1] = (i & 1) ? (dpk[i >> 1] | (d << 16)) : d;
        if (i & 1) __asm__ volatile("" : "+v"(dpk[i >> 1]));
        if (valid) atomicAdd(&sh.u.hist[d], 1u);
      }
    }
  }
  __syncthreads();
  BPC_STAMP(1, 2);
  // The bookkeeping from here to the selection (histogram summary, the
  // candidate list, the threshold) runs at raised wave priority: the
  // workgroups still in it are the youngest on their CU, whose instructions
  // otherwise queue behind the older workgroups' attention passes.  The
  // attention itself runs at the normal priority.
  __builtin_amdgcn_s_setprio(3);
  auto dist_of = [&](int it, int u) -> int {
    const int i = it * KPL + u;
    return (int)((dpk[i >> 1] >> ((i & 1) << 4)) & 0xFFFFu);
  };
  if (score_out) {  // debug output
    int32_t* so = score_out + (size_t)bh * N + n0;
    int kb = wid * KPW + lane * KPL;  // opaque: no per-key offsets are kept from the scoring loop
    __asm__ volatile("" : "+v"(kb));
#pragma unroll
    for (int it = 0; it < NLD; ++it)
#pragma unroll
      for (int u = 0; u < KPL; ++u) {
        const int n = kb + it * KSTEP + u;
        if (n < cnt) so[n] = T - 2 * dist_of(it, u);
      }
  }

  // ---- 2. histogram summary, published --------------------------------
  // the histogram in prefix form per coarse bin (count in [128 (t >> 7), t))
  // << 16 | count at t, and the coarse counts
  for (int seg = threadIdx.x; seg < 1024; seg += NT) {
    const int cbin = seg >> 3, part8 = seg & 7;
    const int fb0 = (cbin << kCoarseShift) + part8 * 16;
    uint32_t cntv[16];
    if (fb0 < NBP) {
      const uint4* hv = reinterpret_cast<const uint4*>(sh.u.hist + fb0);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint4 x = hv[r];
        cntv[4 * r] = x.x, cntv[4 * r + 1] = x.y, cntv[4 * r + 2] = x.z, cntv[4 * r + 3] = x.w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 16; ++e) cntv[e] = 0u;
    }
    int local = 0;
#pragma unroll
    for (int e = 0; e < 16; ++e) local += (int)cntv[e];
    const int incl = group8_inclusive_sum(local);
    if (part8 == 7) sh.coarse[cbin] = (uint32_t)incl;
    if (fb0 < NBP) {
      uint32_t run = (uint32_t)(incl - local);
      uint4* hv = reinterpret_cast<uint4*>(sh.u.hist + fb0);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        uint32_t v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[e] = (run << 16) | cntv[4 * r + e];
          run += cntv[4 * r + e];
        }
        hv[r] = make_uint4(v[0], v[1], v[2], v[3]);
      }
    }
  }
  __syncthreads();
  // wave 0: coarse prefix, the lowest occupied coarse bin, and the fine bins
  // of the slice's k-th key and of its m-th key, m = ceil(k cnt / N) (its
  // share of the budget, its own estimate of the threshold)
  const int mloc = (int)(((int64_t)k * cnt + N - 1) / N);
  if (threadIdx.x < 64) {
    const uint32_t c0 = sh.coarse[2 * lane], c1 = sh.coarse[2 * lane + 1];
    const int x = wave_inclusive_sum((int)(c0 + c1));
    const int ex = x - (int)(c0 + c1);
    sh.cc[2 * lane] = (uint32_t)ex;
    sh.cc[2 * lane + 1] = (uint32_t)ex + c0;
    if (lane == 63) sh.cc[kCoarseBins] = (uint32_t)x;
    auto first_coarse = [&](int need) -> int {
      const int f0 = first_lane(__ballot(ex + (int)c0 >= need)), f1 = first_lane(__ballot(x >= need));
      return min(f0 < 64 ? 2 * f0 : 1 << 30, f1 < 64 ? 2 * f1 + 1 : 1 << 30);
    };
    const int cs = first_coarse(k), cs2 = first_coarse(mloc);
    const int g0 = first_lane(__ballot(c0 != 0u)), g1 = first_lane(__ballot(c1 != 0u));
    auto fine_first = [&](int c, int need) -> int {
      if (c < 0 || c >= kCoarseBins) return NB - 1;
      const int below = __builtin_amdgcn_readlane((c & 1) ? ex + (int)c0 : ex, c >> 1);
      const int t0 = (c << kCoarseShift) + lane, t1 = t0 + 64;
      const uint32_t v0 = (t0 < NBP) ? sh.u.hist[t0] : 0u, v1 = (t1 < NBP) ? sh.u.hist[t1] : 0u;
      const unsigned long long r0 = __ballot(below + (int)(v0 >> 16) + (int)(v0 & 0xFFFFu) >= need);
      const unsigned long long r1 = __ballot(below + (int)(v1 >> 16) + (int)(v1 & 0xFFFFu) >= need);
      return r0 ? (c << kCoarseShift) + first_lane(r0) : r1 ? (c << kCoarseShift) + 64 + first_lane(r1) : NB - 1;
    };
    const int kth_w = fine_first((cnt >= k) ? cs : -1, k);
    const int that_w = fine_first(cs2, mloc);
    if (lane == 0) {
      sh.kth = kth_w;
      sh.that = that_w;
      sh.cmin = min(g0 < 64 ? 2 * g0 : kCoarseBins - 1, g1 < 64 ? 2 * g1 + 1 : kCoarseBins - 1);
    }
  }
  __syncthreads();
  int cand_max;
  {
    // the window: kWinBins distances ending `up` above the slice's estimate t,
    // `up` about six standard deviations of that estimate
    auto cum = [&](int t) -> uint32_t {  // keys with distance <= t
      if (t < 0) return 0u;
      if (t >= NBP) return (uint32_t)cnt;
      const uint32_t v = sh.u.hist[t];
      return sh.cc[t >> kCoarseShift] + (v >> 16) + (v & 0xFFFFu);
    };
    const int that = sh.that;
    const int dens17 = max((int)cum(that + 8) - (int)cum(that - 9), 1);
    const int up = min(max((int)ceilf(6.0f * sqrtf((float)mloc) * 17.0f / (float)dens17), 4), kWinBins - 32);
    const int wbase = max(that + up - (kWinBins - 1), 0);
    // the largest distance on the candidate list: the window's end, at most
    // the slice's k-th smallest distance (T* never exceeds the latter)
    cand_max = min(wbase + kWinBins - 1, sh.kth);
    if (threadIdx.x < kWinBins / 2)
      pub_store(my_pub + 4 + threadIdx.x, cum(wbase + 2 * threadIdx.x) | (cum(wbase + 2 * threadIdx.x + 1) << 16));
    else if (threadIdx.x < kWinBins / 2 + 4) {
      const int j = threadIdx.x - kWinBins / 2;
      const uint32_t hdr[4] = {(uint32_t)wbase, (uint32_t)cand_max, wbase > 0 ? cum(wbase - 1) : 0u,
                               (uint32_t)cnt};
      pub_store(my_pub + j, hdr[j]);
    } else if (threadIdx.x < kWinBins / 2 + 8) {
      const int j = threadIdx.x - kWinBins / 2 - 4;
      const uint32_t mt[4] = {(uint32_t)sh.kth, (uint32_t)sh.cmin, (uint32_t)cnt, 0u};
      pub_store(my_pub + kPubMeta + j, mt[j]);
    }
    for (int c = threadIdx.x; c <= kCoarseBins; c += NT) pub_store(my_pub + kPubCoarse + c, sh.cc[c]);
  }
  BPC_STAMP(1, 5);
  // arrival: every published store of the workgroup is complete first (and
  // every read of the histogram, whose area holds the candidates next)
  stores_complete();
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(bh_sync + 0, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  BPC_STAMP(1, 7);
  // While the other slices finish: the candidates (distance <= cand_max) in
  // key order into the LDS list (at most kRowCache of them).  In key order a
  // lane's KPL keys of one load follow those of the lanes below it: each
  // wavefront counts its own, then writes from a running offset.
  int ncand;
  {
    int c = 0;
#pragma unroll
    for (int it = 0; it < NLD; ++it)
#pragma unroll
      for (int u = 0; u < KPL; ++u) c += dist_of(it, u) <= cand_max;
    c = wave_inclusive_sum(c);
    if (lane == 63) sh.wcnt[wid][0] = c;
  }
  // the write pass re-derives its flags instead of keeping 64 comparisons
#pragma unroll
  for (int i = 0; i < PER / 2; ++i) __asm__ volatile("" : "+v"(dpk[i]));
  __syncthreads();
  {
    int base = 0;
    ncand = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      base += (w < wid) ? sh.wcnt[w][0] : 0;
      ncand += sh.wcnt[w][0];
    }
    if (ncand <= kRowCache) {
      uint32_t* cl = reinterpret_cast<uint32_t*>(sh.u.at.rows);
      int kb = wid * KPW + lane * KPL;  // the lane's first key (opaque: nothing derived from it is precomputed)
      __asm__ volatile("" : "+v"(kb));
#pragma unroll
      for (int it = 0; it < NLD; ++it) {
        int pos = base;
        bool f[KPL];
#pragma unroll
        for (int u = 0; u < KPL; ++u) {
          f[u] = dist_of(it, u) <= cand_max;
          const unsigned long long mk = __ballot(f[u]);
          pos += (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mk >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mk, 0u));
          base += (int)__popcll(mk);
        }
#pragma unroll
        for (int u = 0; u < KPL; ++u)
          if (f[u]) cl[pos++] = ((uint32_t)(kb + it * KSTEP + u) << 16) | (uint32_t)dist_of(it, u);
      }
    }
  }
  if (threadIdx.x == 0) {
    unsigned it = 0;    while (pub_load(bh_sync + 0) < (uint32_t)nslices && ++it < kSpinLimit) __builtin_amdgcn_s_sleep(2);
    sh.flag = it < kSpinLimit;
  }
  // the group's queries for the attention (its own loads, behind the wait)
  if (threadIdx.x < G * kHeadDim / 8) {
    const uint4* qb = reinterpret_cast<const uint4*>(q + ((size_t)b * Hkv * G + (size_t)h * G) * kHeadDim);
    sh.q[threadIdx.x / (kHeadDim / 8)][threadIdx.x % (kHeadDim / 8)] = qb[threadIdx.x];
  }
  __syncthreads();
  BPC_STAMP(1, 3);
  const bool arrived = sh.flag != 0;

  // ---- 3. the threshold T*, this slice's tie quota and offset ---------
  int tstar = 0, take = 0, off = 0, kept = 0;
  bool planned = false, by_window = false;
  if (arrived && nslices <= kWinSlices) {
    // one round over the window records (see the attention kernel above)
    static_assert(2 * kCoarseBins >= kWinBins + 1 && kWinBins + 1 <= 3 * 64, "S(t) fits the scratch and three lanes");
    if (threadIdx.x < 2 * kCoarseBins) (&sh.gsum[0][0])[threadIdx.x] = 0;  // S(t) below (after the copy's barrier)
    // (as 64-bit words: a record is kWinRec / 2 of them, 8-byte aligned)
    constexpr int RW = kWinRec / 2;
    static_assert(kWinRec % 2 == 0 && kPubStride % 2 == 0, "records of whole 64-bit words");
    const int nv = nslices * RW;
    uint64_t* wdst = reinterpret_cast<uint64_t*>(&sh.u.at.win[0][0]);
    auto src = [&](int e) {
      return reinterpret_cast<const uint64_t*>(bh_pub + (size_t)(e / RW) * kPubStride) + e % RW;
    };
    if (nv <= NT)
      copy_published<1>(wdst, nv, src);
    else if (nv <= 2 * NT)
      copy_published<2>(wdst, nv, src);
    else
      copy_published<(kWinSlices * RW + NT - 1) / NT>(wdst, nv, src);
    __syncthreads();
    BPC_NOTE(1, 12, __builtin_amdgcn_s_memrealtime());
    auto cum = [&](int u, int t) -> int {  // base_u - 1 <= t < base_u + kWinBins
      const int j = t - (int)sh.u.at.win[u][0];
      const uint32_t w = sh.u.at.win[u][4 + (max(j, 0) >> 1)];
      return (j < 0) ? (int)sh.u.at.win[u][2] : (int)((j & 1) ? (w >> 16) : (w & 0xFFFFu));
    };
    const int lo = wave_reduce_maxmin<true>(lane < nslices ? (int)sh.u.at.win[lane][0] : 0);
    const int hi = wave_reduce_maxmin<false>(lane < nslices ? (int)sh.u.at.win[lane][1] : (1 << 30));
    // S(t) = sum over the slices of cum_u(t) for t = lo - 1 + i, i < span
    // (at most kWinBins + 1 values): wavefront w adds up slices w, w + NW,
    // ...; lane l holds i = l, l + 64, l + 128, and the wavefronts' sums meet
    // in LDS through atomic adds (integers: the order does not matter).
    // (One thread per t summing every slice waited on two dependent LDS
    // reads per slice: 6.5 us with 64 slices.)
    int* Ssum = &sh.gsum[0][0];
    const int span = lo <= hi ? hi - lo + 2 : 0;
    if (lo <= hi) {
      int a0 = 0, a1 = 0, a2 = 0;
      // the bases and below-window counts of the wavefront's slices, lane v
      // holding slice wid + NW v: read once, then taken by read-lane, so that
      // no LDS read waits on another
      const int uv = wid + NW * lane;
      const int vbase = uv < nslices ? (int)sh.u.at.win[uv][0] : 0;
      const int vbelow = uv < nslices ? (int)sh.u.at.win[uv][2] : 0;
      int v = 0;
#pragma unroll 4
      for (int u = wid; u < nslices; u += NW, ++v) {
        const int base = __builtin_amdgcn_readlane(vbase, v), blw = __builtin_amdgcn_readlane(vbelow, v);
        auto val = [&](int i) -> int {  // cum_u(lo - 1 + i)
          const int j = lo - 1 + i - base;
          const uint32_t w = sh.u.at.win[u][4 + (max(j, 0) >> 1)];
          return j < 0 ? blw : (int)((j & 1) ? (w >> 16) : (w & 0xFFFFu));
        };
        a0 += lane < span ? val(lane) : 0;
        a1 += lane + 64 < span ? val(lane + 64) : 0;
        a2 += lane + 128 < span ? val(lane + 128) : 0;
      }
      if (lane < span) atomicAdd(&Ssum[lane], a0);
      if (lane + 64 < span) atomicAdd(&Ssum[lane + 64], a1);
      if (lane + 128 < span) atomicAdd(&Ssum[lane + 128], a2);
    }
    __syncthreads();
    bool below = false, badt = false;
    const int t = lo - 1 + (int)threadIdx.x;
    if (lo <= hi && t <= hi) {
      const int St = Ssum[threadIdx.x];
      if (t == lo - 1)
        badt = St >= k;
      else
        below = St < k;
      if (t == hi && St < k) badt = true;
    }
    const unsigned long long mbelow = __ballot(below), mbad = __ballot(badt);
    if (lane == 0) sh.red[0][wid] = (int)__popcll(mbelow), sh.red[1][wid] = mbad != 0ull;
    __syncthreads();
    BPC_NOTE(1, 13, __builtin_amdgcn_s_memrealtime());
    int cntlow = 0, bad = lo > hi;
#pragma unroll
    for (int w = 0; w < NW; ++w) cntlow += sh.red[0][w], bad |= sh.red[1][w];
    if (!bad) {
      tstar = lo + cntlow;
      int bu = 0, tu = 0;
      if (lane < nslices) {
        bu = cum(lane, tstar - 1);
        tu = cum(lane, tstar) - bu;
      }
      const int bi = wave_inclusive_sum(bu), ti = wave_inclusive_sum(tu);
      const int below_all = __builtin_amdgcn_readlane(bi, 63);
      const int below_before = __builtin_amdgcn_readlane(bi - bu, s), ties_before = __builtin_amdgcn_readlane(ti - tu, s);
      const int bs = __builtin_amdgcn_readlane(bu, s), ts = __builtin_amdgcn_readlane(tu, s);
      const int need = k - below_all;
      take = max(0, min(ts, need - ties_before));
      off = below_before + min(need, ties_before);
      kept = bs + take;
      planned = by_window = true;
    }
    __syncthreads();  // the window area is reused below
  }
  if (arrived && !planned) {
    // Two exact rounds.  Round 1: the coarse bin c* of the k-th smallest
    // distance from every slice's coarse prefix.
    if (threadIdx.x < kCoarseBins) {
      const int c = threadIdx.x;
      const int gc = sum_published(nslices, [&](int u) { return bh_pub + (size_t)u * kPubStride + kPubCoarse + c + 1; },
                                   [](uint32_t v) { return (int)v; });
      sh.gsum[0][c] = gc;  // keys of all slices with coarse bin <= c
      const unsigned long long mk = __ballot(gc >= k);
      if (lane == 0) sh.red[0][wid] = mk ? first_lane(mk) + 64 * wid : (1 << 30);
    }
    __syncthreads();
    const int cstar = min(min(sh.red[0][0], sh.red[0][1]), kCoarseBins - 1);
    const int below_c = (cstar > 0) ? sh.gsum[0][cstar - 1] : 0;
    // Round 2: this slice's fine bins of c*, counted from its registers and
    // published in prefix form ((count below bin j in c*) << 16 | count at j)
    for (int j = threadIdx.x; j < (1 << kCoarseShift); j += NT) sh.fine[j] = 0u;
    __syncthreads();
#pragma unroll
    for (int it = 0; it < NLD; ++it)
#pragma unroll
      for (int u = 0; u < KPL; ++u) {
        const int d = dist_of(it, u);
        if ((d >> kCoarseShift) == cstar && d < NB) atomicAdd(&sh.fine[d & ((1 << kCoarseShift) - 1)], 1u);
      }
    __syncthreads();
    if (threadIdx.x < 64) {
      const uint32_t a0 = sh.fine[2 * lane], a1 = sh.fine[2 * lane + 1];
      const int x = wave_inclusive_sum((int)(a0 + a1));
      const uint32_t ex = (uint32_t)x - a0 - a1;
      pub_store(my_pub + kPubFine + 2 * lane, (ex << 16) | a0);
      pub_store(my_pub + kPubFine + 2 * lane + 1, ((ex + a0) << 16) | a1);
    }
    stores_complete();
    __syncthreads();
    if (threadIdx.x == 0) {
      __hip_atomic_fetch_add(bh_sync + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      unsigned it = 0;
      while (pub_load(bh_sync + 1) < (uint32_t)nslices && ++it < kSpinLimit) __builtin_amdgcn_s_sleep(2);
      sh.flag = it < kSpinLimit;
    }
    __syncthreads();
    if (sh.flag) {
      // bin j of c*: keys of all slices below it (exc) and up to it (inc)
      if (threadIdx.x < (1 << kCoarseShift)) {
        const int j = threadIdx.x;
        auto at = [&](int u) { return bh_pub + (size_t)u * kPubStride + kPubFine + j; };
        const int exc = sum_published(nslices, at, [](uint32_t v) { return (int)(v >> 16); });
        const int inc = exc + sum_published(nslices, at, [](uint32_t v) { return (int)(v & 0xFFFFu); });
        sh.gsum[1][j] = exc;
        const unsigned long long mk = __ballot(below_c + inc >= k);
        if (lane == 0) sh.red[1][wid] = mk ? first_lane(mk) + 64 * wid : (1 << 30);
      }
      __syncthreads();
      const int jt = min(min(sh.red[1][0], sh.red[1][1]), (1 << kCoarseShift) - 1);
      tstar = min((cstar << kCoarseShift) + jt, NB - 1);
      const int need = k - (below_c + sh.gsum[1][jt]);  // keys at T* to take, over all slices
      // keys below T* and ties at T* of the slices before s (thread u for
      // slice u), and of s itself
      int bl = 0, ti = 0, my_below = 0, my_tie = 0;
      for (int u = threadIdx.x; u <= s; u += NT) {
        const uint32_t* pu = bh_pub + (size_t)u * kPubStride;
        const uint32_t ccu = pub_load(pu + kPubCoarse + cstar), fu = pub_load(pu + kPubFine + jt);
        const int below = (int)ccu + (int)(fu >> 16), tie = (int)(fu & 0xFFFFu);
        if (u < s) {
          bl += below, ti += tie;
        } else {
          my_below = below, my_tie = tie;
        }
      }
      bl = wave_inclusive_sum(bl);
      ti = wave_inclusive_sum(ti);
      if (lane == 63) sh.wave_tot[0][wid] = bl, sh.wave_tot[1][wid] = ti;
      if ((s % NT) == (int)threadIdx.x) sh.red[0][2] = my_below, sh.red[1][2] = my_tie;
      __syncthreads();
      int below_before = 0, ties_before = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) below_before += sh.wave_tot[0][w], ties_before += sh.wave_tot[1][w];
      my_below = sh.red[0][2], my_tie = sh.red[1][2];
      take = max(0, min(my_tie, need - ties_before));
      off = below_before + min(need, ties_before);
      kept = my_below + take;
      planned = true;
      __syncthreads();
    }
  }
  if (!planned) kept = 0;  // a bounded wait ran out: this slice contributes nothing
  kept = max(0, min(kept, k - off));
  BPC_STAMP(1, 4);
  BPC_NOTE(1, 14, by_window ? 1 : 2);

  // ---- 4. selection and attention -----------------------------------
  // A kept key's rank among the slice's kept keys (key order) is (keys below
  // T* before it) + min(ties at T* before it, take).  With the one-round
  // threshold every key at or below T* is a candidate (T* <= cand_max), and
  // the selection reads the candidate list only; otherwise the slice's keys
  // are walked again from the registers.
  if (m > 0)
    for (int i = threadIdx.x; i < SL / 32; i += NT) sh.u.at.sel[i] = 0u;
  int32_t* grow = rows + (size_t)bh * k;  // the (b, h)'s global row list (ranks past the LDS list)
  const bool from_cands = by_window && ncand <= kRowCache;
  if (from_cands) {
    // batches of 4 NT candidates: their ranks from one block scan of the
    // packed (ties << 16 | below) counts; the kept keys are written over the
    // list itself (a kept candidate's rank never exceeds its position, and a
    // batch is read before the scan's barrier)
    uint32_t* cl = reinterpret_cast<uint32_t*>(sh.u.at.rows);
    int nkept = 0, tie_seen = 0, sbuf = 0;
    __syncthreads();  // the candidate list (and a cleared bitmap) visible to all
    for (int base = 0; base < ncand; base += 4 * NT) {
      const int nvalid = ncand - base - (int)threadIdx.x * 4;
      uint32_t cv[4];
      int nb = 0, nt = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        cv[e] = (e < nvalid) ? cl[base + threadIdx.x * 4 + e] : 0xFFFFFFFFu;
        const int d = (int)(cv[e] & 0xFFFFu);
        nb += (e < nvalid) && d < tstar;
        nt += (e < nvalid) && d == tstar;
      }
      int tot;
      const int pre = block_exclusive_scan_bits<NT, 0x70007u>((nt << 16) | nb, sh.wave_tot, sbuf, tot);
      sbuf ^= 1;
      int tie_rank = tie_seen + (pre >> 16);
      int rank = nkept + (pre & 0xFFFF) + max(0, min(tie_rank, take) - min(tie_seen, take));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int d = (e < nvalid) ? (int)(cv[e] & 0xFFFFu) : (1 << 30);
        bool keep = d < tstar;
        if (d == tstar) {
          keep = tie_rank < take;
          ++tie_rank;
        }
        if (keep && rank < kept) {
          const int kin = (int)(cv[e] >> 16);
          sh.u.at.rows[rank] = n0 + kin;
          if (idx_out) idx_out[(size_t)bh * k + off + rank] = n0 + kin;
          if (m > 0) atomicOr(&sh.u.at.sel[kin >> 5], 1u << (kin & 31));
        }
        rank += keep;
      }
      nkept += (tot & 0xFFFF) + max(0, min(tie_seen + (tot >> 16), take) - min(tie_seen, take));
      tie_seen += tot >> 16;
    }
  } else {
    int nb = 0, nt = 0;
#pragma unroll
    for (int it = 0; it < NLD; ++it)
#pragma unroll
      for (int u = 0; u < KPL; ++u) {
        const int d = dist_of(it, u);
        nb += d < tstar;
        nt += d == tstar;
      }
    nb = wave_inclusive_sum(nb);
    nt = wave_inclusive_sum(nt);
    if (lane == 63) sh.wcnt[wid][0] = nb, sh.wcnt[wid][1] = nt;
    __syncthreads();
  int wb0 = 0, wt0 = 0;  // keys below T* and ties at T* in the wavefronts before this one
#pragma unroll
  for (int w = 0; w < NW; ++w)
    if (w < wid) wb0 += sh.wcnt[w][0], wt0 += sh.wcnt[w][1];
  // The walk writes LDS only (global stores in its fully unrolled loop make
  // the compiler spill): the rows of ranks [lo, lo + kRowCache) into the LDS
  // list and the selection bitmap.  Windows past the first are walked first
  // and copied out to the (b, h)'s global row list; the first stays in LDS.
  const int nwin = max(1, (kept + kRowCache - 1) / kRowCache);
  for (int wnd = nwin - 1; wnd >= 0; --wnd) {
    const int lo = wnd * kRowCache;
    int wb = wb0, wt = wt0;
    // the lane's first key, opaque to the compiler: values derived from the
    // keys are computed where they are used, not hoisted out of this loop
    // for all 64 keys (which would spill)
    int kb = wid * KPW + lane * KPL;
    __asm__ volatile("" : "+v"(kb));
#pragma unroll
    for (int it = 0; it < NLD; ++it) {
      // the keys of one load of the wavefront in ascending order are (lane,
      // u): a lane's KPL keys follow the keys of the lanes below it
      bool fb[KPL], ft[KPL];
      int rb = wb, rt = wt, tb = 0, tt = 0;
#pragma unroll
      for (int u = 0; u < KPL; ++u) {
        const int d = dist_of(it, u);
        fb[u] = d < tstar;
        ft[u] = d == tstar;
        const unsigned long long mb = __ballot(fb[u]), mt = __ballot(ft[u]);
        rb += (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mb >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mb, 0u));
        rt += (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mt >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mt, 0u));
        tb += (int)__popcll(mb);
        tt += (int)__popcll(mt);
      }
      wb += tb;
      wt += tt;
      if (tb + tt == 0) continue;  // uniform over the wavefront
#pragma unroll
      for (int u = 0; u < KPL; ++u) {
        const bool keep = fb[u] || (ft[u] && rt < take);
        const int rank = rb + min(rt, take);
        if (keep && rank < kept) {
          const int kin = kb + it * KSTEP + u;
          if (m > 0 && wnd == 0) atomicOr(&sh.u.at.sel[kin >> 5], 1u << (kin & 31));
          if (rank >= lo && rank < lo + kRowCache) sh.u.at.rows[rank - lo] = n0 + kin;
        }
        rb += fb[u];
        rt += ft[u];
      }
    }
    __syncthreads();
    if (wnd > 0) {
      const int nr = min(kRowCache, kept - lo);
      for (int r = threadIdx.x; r < nr; r += NT) {
        const int key = sh.u.at.rows[r];
        grow[off + lo + r] = key;
        if (idx_out) idx_out[(size_t)bh * k + off + lo + r] = key;
      }
      __syncthreads();
    }
  }
  if (idx_out)
    for (int r = threadIdx.x; r < min(kept, kRowCache); r += NT) idx_out[(size_t)bh * k + off + r] = sh.u.at.rows[r];
  }
  __syncthreads();  // the kept rows and the selection bitmap are complete
  int extra = 0;
  if (m > 0) {
    // S_err entries of this slice the hash selection did not take, in S_err
    // order (ascending keys), ranked kept + (their position among them); the
    // ones past the LDS list are found again from S_err when they are read
    const int32_t* se = serr + b * sS_b + h * sS_h;
    int sbuf = 0;
    for (int base = 0; base < m; base += 4 * NT) {
      int key[4], add[4], na = 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = base + 4 * (int)threadIdx.x + u;
        key[u] = (j < m) ? se[j] : -1;
        const int kin = key[u] - n0;
        const bool here = key[u] >= n0 && kin < cnt;
        add[u] = here && !((sh.u.at.sel[kin >> 5] >> (kin & 31)) & 1u);
        if (added_out) {
          const bool outside = j < m && (key[u] < 0 || key[u] >= N);
          if (here || (outside && s == 0)) added_out[(size_t)bh * m + j] = add[u];
        }
        na += add[u];
      }
      int tot;
      int pos = kept + extra + block_exclusive_scan_bits<NT, 0x7u>(na, sh.wave_tot, sbuf, tot);
      sbuf ^= 1;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (add[u]) {
          if (pos < kRowCache) sh.u.at.rows[pos] = key[u];
          ++pos;
        }
      extra += tot;
    }
    __syncthreads();
  }
  const int nrows = kept + extra;
  float mx = -INFINITY, ls = 0.f;  // running (max, sum) of query head lane % 16 (lanes below G)
  f32x4_t acc[8];
#pragma unroll
  for (int T = 0; T < 8; ++T) acc[T] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  char* vt = reinterpret_cast<char*>(&sh.u.at.win[0][0]) + wid * kVtWaveBytes;  // free once T* is known
  const char* Kh = reinterpret_cast<const char*>(K + b * sK_b + h * sK_h);
  const char* Vh = reinterpret_cast<const char*>(V + b * sV_b + h * sV_h);
  const uint32_t kstride = (uint32_t)sK_n * 2u, vstride = (uint32_t)sV_n * 2u;
  BPC_STAMP(1, 8);
  __builtin_amdgcn_s_setprio(0);
  if (nrows <= kRowCache) {
    for (int q0 = wid * kAttnRows; q0 < nrows; q0 += NW * kAttnRows) {
      const int nr = min(kAttnRows, nrows - q0);
      const int c16 = lane & 15, r4 = lane >> 4;
      const int kc = sh.u.at.rows[q0 + c16];
      const int4 v4 = *reinterpret_cast<const int4*>(sh.u.at.rows + q0 + 4 * r4);
      const uint32_t rk = c16 < nr ? (uint32_t)kc : 0u;
      uint32_t rv[4];
      rv[0] = 4 * r4 + 0 < nr ? (uint32_t)v4.x : 0u;
      rv[1] = 4 * r4 + 1 < nr ? (uint32_t)v4.y : 0u;
      rv[2] = 4 * r4 + 2 < nr ? (uint32_t)v4.z : 0u;
      rv[3] = 4 * r4 + 3 < nr ? (uint32_t)v4.w : 0u;
      attend_pass_mfma<G>(rk, rv, nr, sh.q, vt, Kh, kstride, Vh, vstride, scale_log2, mx, ls, acc);
    }
  } else {
    // more rows than the LDS list holds: rank r >= kRowCache is at
    // grow[off + r] (a kept key) or is an extra row of the safeguard (found
    // again from the S_err order)
    const int32_t* se = (m > 0) ? serr + b * sS_b + h * sS_h : nullptr;
    int jlo = 0;  // S_err entries before this slice's keys (S_err is ascending)
    if (m > 0) {
      int c = 0;
      for (int j = threadIdx.x; j < m; j += NT) c += se[j] < n0;
      c = wave_inclusive_sum(c);
      if (lane == 63) sh.red[0][wid] = c;
      __syncthreads();
#pragma unroll
      for (int w = 0; w < NW; ++w) jlo += sh.red[0][w];
      __syncthreads();
    }
    auto rank_row = [&](int r) -> uint32_t {
      if (r >= nrows) return 0u;
      if (r < kRowCache) return (uint32_t)sh.u.at.rows[r];
      if (r < kept) return (uint32_t)grow[off + r];
      // the (r - kept)-th added S_err entry of this slice: scan from jlo
      int want = r - kept;
      for (int j = jlo; j < m; ++j) {
        const int key = se[j];
        const int kin = key - n0;
        if (key < n0 || kin >= cnt) break;
        if (!((sh.u.at.sel[kin >> 5] >> (kin & 31)) & 1u) && want-- == 0) return (uint32_t)key;
      }
      return 0u;
    };
    for (int q0 = wid * kAttnRows; q0 < nrows; q0 += NW * kAttnRows) {
      const int nr = min(kAttnRows, nrows - q0);
      const int c16 = lane & 15, r4 = lane >> 4;
      const uint32_t rk = c16 < nr ? rank_row(q0 + c16) : 0u;
      uint32_t rv[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) rv[t] = 4 * r4 + t < nr ? rank_row(q0 + 4 * r4 + t) : 0u;
      attend_pass_mfma<G>(rk, rv, nr, sh.q, vt, Kh, kstride, Vh, vstride, scale_log2, mx, ls, acc);
    }
  }
  __syncthreads();  // the rows are read before the partial reuses their area
  BPC_STAMP(1, 9);

  // ---- 5. the partial, published; the last slice of (b, h) merges -----
  float* my_part = part + sl * G * (kHeadDim + 2);
  float Mx[G], Ls[G];
  lane_stats<G>(mx, ls, Mx, Ls);
  write_partial_tiles<G, true>(sh.u.o, sh.st, Mx, Ls, acc, my_part);
  stores_complete();
  __syncthreads();
  if (threadIdx.x == 0)
    sh.flag = __hip_atomic_fetch_add(bh_sync + 2, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
              (uint32_t)(nslices - 1);
  __syncthreads();
  if (!sh.flag) return;
  const float* pbh = part + (size_t)bh * nslices * G * (kHeadDim + 2);
  const size_t cstride = (size_t)G * (kHeadDim + 2);
  if (L != 32 && nslices <= 64) {
    // The merge, up to 64 slices (and L >= 64: at L = 32 the extra registers
    // spill elsewhere in the kernel): per query head (one wavefront, lane u =
    // slice u) the common maximum, each slice's weight exp2(max_u - M) and
    // the weighted sum of the slices' sums (a butterfly, the same in every
    // lane); then each thread one pair of output coordinates, summed over
    // the slices in ascending order with every load of a batch in flight.
    float* wts = reinterpret_cast<float*>(&sh.u.hist[0]);  // [64][G] weights, then [G] totals
    float* tot = wts + 64 * G;
    for (int g = wid; g < G; g += NW) {
      float m = -INFINITY, l = 0.f;
      if (lane < nslices) {
        const uint64_t v =
            pub_load64(reinterpret_cast<const uint64_t*>(pbh + (size_t)lane * cstride + (size_t)g * (kHeadDim + 2)));
        m = __uint_as_float((uint32_t)v), l = __uint_as_float((uint32_t)(v >> 32));
      }
      float M = m;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) M = fmaxf(M, __shfl_xor(M, o, 64));
      const float w = (m == -INFINITY) ? 0.f : exp2f(m - M);
      float sum = w * l;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) sum += __shfl_xor(sum, o, 64);
      wts[lane * G + g] = w;
      if (lane == 0) tot[g] = sum;
    }
    __syncthreads();
    for (int e = threadIdx.x; e < G * (kHeadDim / 2); e += NT) {
      const int g = e / (kHeadDim / 2), d2 = e % (kHeadDim / 2);
      const float* pg = pbh + (size_t)g * (kHeadDim + 2) + 2 + 2 * d2;
      float a0 = 0.f, a1 = 0.f;
      constexpr int MB = 16;  // loads in flight
      for (int u0 = 0; u0 < nslices; u0 += MB) {
        uint64_t v[MB];
#pragma unroll
        for (int j = 0; j < MB; ++j)
          v[j] = (u0 + j < nslices) ? pub_load64(reinterpret_cast<const uint64_t*>(pg + (size_t)(u0 + j) * cstride)) : 0u;
#pragma unroll
        for (int j = 0; j < MB; ++j)
          if (u0 + j < nslices) {
            const float w = wts[(u0 + j) * G + g];
            a0 = fmaf(w, __uint_as_float((uint32_t)v[j]), a0);
            a1 = fmaf(w, __uint_as_float((uint32_t)(v[j] >> 32)), a1);
          }
      }
      float* op = out + ((size_t)b * Hkv * G + (size_t)h * G + g) * kHeadDim + 2 * d2;
      op[0] = a0 / tot[g];
      op[1] = a1 / tot[g];
    }
  } else
  // the merge, more than 64 slices: every slice's (max, sum) per query head
  // with each output coordinate, rescaled batch by batch of eight slices
  for (int e = threadIdx.x; e < G * kHeadDim; e += NT) {
    const int g = e / kHeadDim, d = e % kHeadDim;
    float Mg = -INFINITY, lsum = 0.f, acc = 0.f;
    for (int u0 = 0; u0 < nslices; u0 += 8) {
      float mt[8], lt[8], ot[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float* pc = pbh + (size_t)min(u0 + j, nslices - 1) * cstride + (size_t)g * (kHeadDim + 2);
        mt[j] = __uint_as_float(pub_load(reinterpret_cast<const uint32_t*>(pc)));
        lt[j] = __uint_as_float(pub_load(reinterpret_cast<const uint32_t*>(pc) + 1));
        ot[j] = __uint_as_float(pub_load(reinterpret_cast<const uint32_t*>(pc) + 2 + d));
      }
      float mb = -INFINITY;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (u0 + j >= nslices) mt[j] = -INFINITY;
        mb = fmaxf(mb, mt[j]);
      }
      const float Mn = fmaxf(Mg, mb);
      if (Mn == -INFINITY) continue;
      const float f = (Mg == -INFINITY) ? 0.f : exp2f(Mg - Mn);
      lsum *= f, acc *= f;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float w = (mt[j] == -INFINITY) ? 0.f : exp2f(mt[j] - Mn);
        lsum = fmaf(lt[j], w, lsum);
        acc = fmaf(ot[j], w, acc);
      }
      Mg = Mn;
    }
    out[((size_t)b * Hkv * G + (size_t)h * G + g) * kHeadDim + d] = acc / lsum;
  }
  // every slice of (b, h) has passed every wait: the counters and the shared
  // query rows go back to zero
  if (threadIdx.x < 3) __hip_atomic_store(bh_sync + threadIdx.x, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (nslices > 1 && threadIdx.x < L) pub_store64(xq_of() + threadIdx.x, 0u);
  BPC_STAMP(1, 10);
}

// ---------------------------------------------------------------------------
// Launch sequence (all on the caller's stream): score (with the query
// packing) -> attend -> merge.
// ---------------------------------------------------------------------------
template <int L>
static hipError_t launch_decode_L(const DecodeArgs& a, const DecodeLayout& lay) {
  const int BH = a.B * a.Hkv;
  uint32_t* cand = reinterpret_cast<uint32_t*>(a.ws + lay.off_cand);
  uint32_t* meta = reinterpret_cast<uint32_t*>(a.ws + lay.off_meta);
  uint32_t* hist_fine = reinterpret_cast<uint32_t*>(a.ws + lay.off_hist_fine);
  uint32_t* hist_cc = reinterpret_cast<uint32_t*>(a.ws + lay.off_hist_cc);
  uint32_t* win = reinterpret_cast<uint32_t*>(a.ws + lay.off_win);
  float* part = reinterpret_cast<float*>(a.ws + lay.off_part);
  uint32_t* qcode = reinterpret_cast<uint32_t*>(a.ws + lay.off_qcode);
  const float scale_log2 = a.sm_scale * 1.4426950408889634f;
  hipStream_t st = a.stream;
  auto mark = [&](int i) {
    if (a.events) (void)hipEventRecord(a.events[i], st);
  };
  const int nwg = BH * lay.nslices;
  // the one-round threshold reads the window records of at most kWinSlices slices
  const int win_ok = lay.nslices <= kWinSlices;

  mark(0);
  score_kernel<L, true><<<nwg, kScoreThreads, 0, st>>>(a.q, a.P, a.sP_b, a.sP_h, lay.G, qcode, a.qcode_out, a.codes,
                                                     a.sC_b, a.sC_h, BH, a.Hkv, a.N, a.k, lay.nslices, cand, meta,
                                                     hist_fine, hist_cc, win, a.score_out);
  // slices of the other kind: a ragged last slice, or codes whose head or
  // batch stride is not a multiple of four words (the base is 16-byte aligned)
  if (a.N % kSlice != 0 || (a.sC_b * 4) % 16 != 0 || (a.sC_h * 4) % 16 != 0)
    score_kernel<L, false><<<nwg, kScoreThreads, 0, st>>>(a.q, a.P, a.sP_b, a.sP_h, lay.G, qcode, a.qcode_out,
                                                          a.codes, a.sC_b, a.sC_h, BH, a.Hkv, a.N, a.k, lay.nslices,
                                                          cand, meta, hist_fine, hist_cc, win, a.score_out);
  mark(1);
  switch (lay.G) {
#define BPC_ATTEND_CASE(GG)                                                                                     \
  case GG:                                                                                                      \
    attend_kernel<GG><<<nwg, kAttnThreads, 0, st>>>(a.N, a.k, L, BH, a.Hkv, lay.nslices, win_ok, cand, meta,    \
                                                    hist_fine, hist_cc, win, a.codes, a.sC_b, a.sC_h, qcode,      \
                                                    a.idx_out, a.serr, a.sS_b, a.sS_h, a.m, a.added_out, a.q, a.K, \
                                                    a.sK_b, a.sK_h, a.sK_n, a.V, a.sV_b, a.sV_h, a.sV_n,          \
                                                    scale_log2, part);                                            \
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
  mark(2);
  merge_kernel<<<a.B * a.Hq, kHeadDim, 0, st>>>(a.Hkv, lay.G, lay.nslices, part, a.out);
  mark(3);
  return hipGetLastError();
}

#ifdef BPC_TRACE
extern "C" int bpc_trace_buffer(void* buf) {
  return hipMemcpyToSymbol(HIP_SYMBOL(g_trace), &buf, sizeof(buf)) == hipSuccess ? 0 : -1;
}
#endif

hipError_t launch_dense(const DenseArgs& a) {
  const int BH = a.B * a.Hkv, G = a.Hq / a.Hkv;
  const int nchunks = (a.N + kSlice - 1) / kSlice;
  const int nwg = BH * nchunks;
  float* part = reinterpret_cast<float*>(a.ws);
  const float scale_log2 = a.sm_scale * 1.4426950408889634f;
  switch (G) {
#define BPC_DENSE_CASE(GG)                                                                                         \
  case GG:                                                                                                         \
    dense_kernel<GG><<<nwg, kAttnThreads, 0, a.stream>>>(a.N, a.Hkv, nchunks, a.q, a.K, a.sK_b, a.sK_h, a.sK_n, a.V, \
                                                         a.sV_b, a.sV_h, a.sV_n, scale_log2, part);               \
    break;
    BPC_DENSE_CASE(1)
    BPC_DENSE_CASE(2)
    BPC_DENSE_CASE(4)
    BPC_DENSE_CASE(8)
    BPC_DENSE_CASE(16)
#undef BPC_DENSE_CASE
    default:
      break;
  }
  merge_kernel<<<a.B * a.Hq, kHeadDim, 0, a.stream>>>(a.Hkv, G, nchunks, part, a.out);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// The fused path: chosen when the grid fits on the device at once (the
// occupancy of the kernel instance times the compute units), cached per
// device, kernel instance and process.
// ---------------------------------------------------------------------------
static std::atomic<int> g_decode_path{0};
void decode_set_path(int path) { g_decode_path.store(path); }

// compute units of the current device (cached per device; at least 1)
static int device_cu_count() {
  constexpr int kDevices = 64;
  static std::atomic<int> cus[kDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kDevices) return 256;
  int c = cus[dev].load();
  if (c == 0) {
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || c < 1) c = 256;
    cus[dev].store(c);
  }
  return c;
}

template <int L, int G, int SL>
static int fused_capacity() {
  constexpr int kDevices = 64;
  static std::atomic<int> cap[kDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kDevices) return 0;
  int c = cap[dev].load();
  if (c == 0) {
    int nb = 0, ncu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fused_decode_kernel<L, G, SL>, kFusedThreads, 0) != hipSuccess ||
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;  // (the error is reported by the launch path)
    c = max(nb * ncu, 0) + 1;  // stored + 1 so that 0 means "not queried"
    cap[dev].store(c);
  }
  return c - 1;
}

template <int L, int SL>
static int fused_capacity_L(int G) {
  switch (G) {
    case 1: return fused_capacity<L, 1, SL>();
    case 2: return fused_capacity<L, 2, SL>();
    case 4: return fused_capacity<L, 4, SL>();
    case 8: return fused_capacity<L, 8, SL>();
    case 16: return fused_capacity<L, 16, SL>();
    default: return 0;
  }
}

// the small-slice instances: code lengths 32 and 64, groups of up to 8
static bool small_slices_built(int L, int G) { return L != 128 && G <= 8; }

template <int SL>
static int fused_capacity_small(int L, int G) {
  if (!small_slices_built(L, G)) return 0;
  if (L == 32) {
    switch (G) {
      case 1: return fused_capacity<32, 1, SL>();
      case 2: return fused_capacity<32, 2, SL>();
      case 4: return fused_capacity<32, 4, SL>();
      default: return fused_capacity<32, 8, SL>();
    }
  }
  switch (G) {
    case 1: return fused_capacity<64, 1, SL>();
    case 2: return fused_capacity<64, 2, SL>();
    case 4: return fused_capacity<64, 4, SL>();
    default: return fused_capacity<64, 8, SL>();
  }
}

static int fused_capacity_of(int L, int G, int SL) {
  if (SL == kSliceSmall) return fused_capacity_small<kSliceSmall>(L, G);
  if (SL == kSliceMid) return fused_capacity_small<kSliceMid>(L, G);
  if (SL != kSlice) return 0;
  return L == 32 ? fused_capacity_L<32, kSlice>(G) : L == 64 ? fused_capacity_L<64, kSlice>(G) : fused_capacity_L<128, kSlice>(G);
}

int decode_fused_slice(int B, int Hq, int Hkv, int N, int L) {
  const int path = g_decode_path.load();
  if (path == 1 || Hkv < 1 || Hq % Hkv || (int64_t)B * Hkv > kFusedMaxBH) return 0;
  const int G = Hq / Hkv;
  // Smaller slices where the 16384-key grid leaves the device mostly idle:
  // the smallest size whose grid stays within two workgroups per compute
  // unit (measured: batch 8 x 8 heads x 65536 keys 37.8 -> 34.7 us on 8192
  // keys, 40.9 on 4096; batch 1 x 8 heads x 32768 keys 35.4 -> 25.3 us on
  // 4096), fits on the device at once and keeps each (b, h) within the
  // one-round threshold's 64 slices.
  if (path == 0 && small_slices_built(L, G)) {
    const int64_t ncu = device_cu_count();
    for (const int sl : {kSliceSmall, kSliceMid}) {
      const int64_t ns = (N + sl - 1) / sl;
      const int64_t nwg = (int64_t)B * Hkv * ns;
      if (ns > 1 && ns <= kWinSlices && nwg <= 2 * ncu && nwg <= fused_capacity_of(L, G, sl)) return sl;
    }
  }
  const int64_t nwg = (int64_t)B * Hkv * ((N + kSlice - 1) / kSlice);
  return nwg <= fused_capacity_of(L, G, kSlice) ? kSlice : 0;
}

template <int L, int SL>
static hipError_t launch_fused_L(const DecodeArgs& a, const DecodeLayout& lay) {
  const int BH = a.B * a.Hkv;
  const int nwg = BH * lay.nslices;
  uint32_t* sync = reinterpret_cast<uint32_t*>(a.ws + lay.off_sync);
  uint32_t* pub = reinterpret_cast<uint32_t*>(a.ws + lay.off_pub);
  float* part = reinterpret_cast<float*>(a.ws + lay.off_part);
  int32_t* rows = reinterpret_cast<int32_t*>(a.ws + lay.off_rows);
  const float scale_log2 = a.sm_scale * 1.4426950408889634f;
  const int ncu = device_cu_count();
  hipStream_t st = a.stream;
  auto mark = [&](int i) {
    if (a.events) (void)hipEventRecord(a.events[i], st);
  };
  mark(0);
  switch (lay.G) {
#define BPC_FUSED_CASE(GG)                                                                                          \
  case GG:                                                                                                          \
    if constexpr (SL == kSlice || GG <= 8)                                                                          \
      fused_decode_kernel<L, GG, SL><<<nwg, kFusedThreads, 0, st>>>(                                                \
          a.q, a.P, a.sP_b, a.sP_h, a.codes, a.sC_b, a.sC_h, a.K, a.sK_b, a.sK_h, a.sK_n, a.V, a.sV_b, a.sV_h,      \
          a.sV_n, BH, a.Hkv, a.N, a.k, lay.nslices, scale_log2, sync, pub, part, rows, a.out, a.idx_out,            \
          a.score_out, a.qcode_out, a.serr, a.sS_b, a.sS_h, a.m, a.added_out, ncu);                                  \
    break;
    BPC_FUSED_CASE(1)
    BPC_FUSED_CASE(2)
    BPC_FUSED_CASE(4)
    BPC_FUSED_CASE(8)
    BPC_FUSED_CASE(16)
#undef BPC_FUSED_CASE
    default:
      break;
  }
  mark(1);
  mark(2);
  mark(3);
  return hipGetLastError();
}

hipError_t launch_decode(const DecodeArgs& a, const DecodeLayout& lay) {
  if (lay.fused) {
    if (lay.slice == kSliceSmall) return a.L == 32 ? launch_fused_L<32, kSliceSmall>(a, lay) : launch_fused_L<64, kSliceSmall>(a, lay);
    if (lay.slice == kSliceMid) return a.L == 32 ? launch_fused_L<32, kSliceMid>(a, lay) : launch_fused_L<64, kSliceMid>(a, lay);
    switch (a.L) {
      case 32: return launch_fused_L<32, kSlice>(a, lay);
      case 64: return launch_fused_L<64, kSlice>(a, lay);
      default: return launch_fused_L<128, kSlice>(a, lay);
    }
  }
  switch (a.L) {
    case 32: return launch_decode_L<32>(a, lay);
    case 64: return launch_decode_L<64>(a, lay);
    default: return launch_decode_L<128>(a, lay);
  }
}

}  // namespace bpc
