// Internal declarations shared by the HIP translation units of libbpc.
//
// Every file of the library is compiled with -ffp-contract=off: the
// sign-deciding sums must round after each multiply and each add, exactly
// as the fixed-order arithmetic documented in include/bpc.h prescribes.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/bpc.h"

namespace bpc {

constexpr int kHeadDim = 128;

// ---- decode tiling ---------------------------------------------------------
// One scoring workgroup owns a slice of kSlice consecutive keys of one
// (sequence, KV head); the slice's distances stay in registers and its
// histogram in LDS.  At most kMaxSlices slices per (sequence, KV head).
constexpr int kSlice = 16384;
// The fused decode path also runs on slices of 8192 or 4096 keys when the
// kSlice grid would leave most of the device idle (code lengths 32 and 64,
// groups of up to 8 query heads).
constexpr int kSliceMid = 8192;
constexpr int kSliceSmall = 4096;
constexpr int kScoreThreads = 512;  // scoring workgroup: 32 keys per thread
constexpr int kMaxSlices = 1024;
// One attention workgroup per slice keeps its selected candidates, read in
// batches of kCandBatch, and gathers their rows with four wavefronts.
constexpr int kAttnThreads = 256;
constexpr int kCandBatch = 1024;
constexpr int kCoarseShift = 7;  // coarse histogram bin = distance >> 7
constexpr int kCoarseBins = 128;
constexpr int kMaxGroup = 16;  // query heads per KV head

// Weighted Hamming distances lie in [0, 127 L].
__host__ __device__ constexpr int dist_bins(int L) { return 127 * L + 1; }
// Per-slice fine histogram: one u32 per distance bin, (count of keys with
// distance in [128 * (t >> 7), t)) << 16 | (count at t); stride padded to
// 16 bytes.  Per-slice coarse prefix: 129 u32 (keys with distance < 128 c),
// stride kCoarseStride.
__host__ __device__ constexpr int fine_stride(int L) { return (dist_bins(L) + 3) & ~3; }
constexpr int kCoarseStride = 132;
// Per-slice window record: header [4] u32 (base, cand_max, keys with
// distance < base, keys in the slice), then kWinBins cumulative counts (keys
// with distance <= base + j) as u16 pairs.  The window ends a few standard
// deviations above the slice's own estimate of the threshold (its
// ceil(k cnt / N)-th smallest distance), and cand_max <= base + kWinBins - 1
// is the largest distance on the slice's candidate list.
constexpr int kWinBins = 128;
constexpr int kWinRec = 4 + kWinBins / 2;  // u32 per record
constexpr int kWinSlices = 64;             // slices per (b, h) the one-round threshold handles

// Fused single-kernel decode (all slices of the grid resident at once): per
// (b, h) kFusedSyncWords u32 of arrival counters (zero between calls), per
// slice kFusedPubWords u32 of published threshold data and G (max, sum,
// o[128]) partials, per (b, h) a row list of k ints for rows past the LDS list.
constexpr int kFusedSyncWords = 16;
constexpr int kFusedPubWords = kWinRec + 4 + kCoarseStride + 128;
// The counters sit in a fixed region at the start of every decode workspace
// (either path), for up to kFusedMaxBH (b, h) pairs, followed by the
// projected query rows the slices of a (b, h) share (kFusedMaxL fp64 rows per
// (b, h), zero while no step runs); the three-launch path never writes the
// region, so it stays zero once zeroed.  (More (b, h) pairs than the fused
// grid's workgroups never take the fused path anyway.)
constexpr int kFusedMaxBH = 1024;
constexpr int kFusedMaxL = 128;
constexpr size_t kSyncCounterBytes = (size_t)kFusedMaxBH * kFusedSyncWords * sizeof(uint32_t);
constexpr size_t kSyncRegionBytes = kSyncCounterBytes + (size_t)kFusedMaxBH * kFusedMaxL * sizeof(uint64_t);

// ---- build tiling ----------------------------------------------------------
constexpr int kBuildGroups = 2;                  // groups of 64 keys per build workgroup
constexpr int kBuildThreads = 256 * kBuildGroups;  // four wavefronts (coordinate blocks) per group
constexpr int kBuildChunk = 64 * kBuildGroups;     // keys per workgroup (one chunk of the row tree)
#ifndef BPC_BUILD_CKPT_PERIOD
#define BPC_BUILD_CKPT_PERIOD 16
#endif
// bits between stored fp64 residuals when the build keeps a checkpoint
constexpr int kBuildCkptPeriod = BPC_BUILD_CKPT_PERIOD;
// chunk sums folded per workgroup before the per-(b, h) reduction, when a
// (b, h) has more than 8 such blocks of chunks
constexpr int kBuildFold = 32;

// ---- workspace layouts -----------------------------------------------------
// Decode, per slice sl = (b Hkv + h) nslices + s: candidates [kSlice] u32
// (key-in-slice << 16 | distance), meta [4] u32 (kth_s, lowest occupied
// coarse bin, candidate count, largest candidate distance), fine histogram
// [fine_stride] u32, coarse
// prefix [kCoarseStride] u32, window record [kWinRec] u32 and G partials of
// (max, sum, o[128]) fp32; per (b, h) the packed query (8 W plane words,
// then sum |p|; stride kQcodeStride).  When a slice keeps more rows than its
// LDS list holds, the attention kernel writes them over the slice's own
// candidate area (a kept entry's rank never exceeds its position there).
constexpr int kQcodeStride = 64;
// Both paths begin with the counter region (kSyncRegionBytes, zero before
// the first call on the workspace, left zero by every call).  The fused
// path's workspace (fused = true) then holds arrival counters [B Hkv]
// [kFusedSyncWords] u32 (inside the region), published records [slices]
// [kFusedPubWords] u32, partials [slices][G][130] fp32 and row lists
// [B Hkv][k] int32.
struct DecodeLayout {
  bool fused;
  int slice;  // keys per slice (kSlice, or kSliceMid / kSliceSmall on the fused path)
  int nslices, G, W;
  size_t off_cand, off_meta, off_hist_fine, off_hist_cc, off_win, off_part, off_qcode, total;
  size_t off_sync, off_pub, off_rows;
};

struct BuildLayout {
  int nchunks;
  int nfold;  // aligned blocks of kBuildFold chunks folded first, or 0
  size_t off_part, off_fold, off_p64, off_g64, total;
  size_t off_ck, total_ck;  // the residual checkpoint, when the workspace holds one
};

DecodeLayout decode_layout(int B, int Hq, int Hkv, int N, int L, int k);
// Keys per slice when the current device runs the decode step as the single
// fused launch (every slice's workgroup resident at once), else 0.
int decode_fused_slice(int B, int Hq, int Hkv, int N, int L);
inline bool decode_fused_ok(int B, int Hq, int Hkv, int N, int L) { return decode_fused_slice(B, Hq, Hkv, N, L) != 0; }
// 0: automatic; 1: always the three-launch path; 2: the fused path only on
// slices of kSlice keys (for comparisons)
void decode_set_path(int path);
BuildLayout build_layout(int B, int Hkv, int N, int L);

// ---- launchers (enqueue only; arguments already validated) ---------------
struct DecodeArgs {
  const uint16_t* q;
  const uint16_t* K;
  int64_t sK_b, sK_h, sK_n;
  const uint16_t* V;
  int64_t sV_b, sV_h, sV_n;
  const uint32_t* codes;
  int64_t sC_b, sC_h;
  const float* P;
  int64_t sP_b, sP_h;
  int B, Hq, Hkv, N, L, k;
  float sm_scale;
  float* out;
  int32_t* idx_out;
  int32_t* score_out;
  uint32_t* qcode_out;
  const int32_t* serr;  // error-aware safeguard: [B, Hkv, m] ascending, or nullptr
  int64_t sS_b, sS_h;
  int m;
  int32_t* added_out;
  char* ws;
  hipStream_t stream;
  hipEvent_t const* events;  // BPC_DECODE_STAGES + 1 handles, or nullptr
};

hipError_t launch_decode(const DecodeArgs& a, const DecodeLayout& lay);

// dense decode attention (full softmax over all N keys), the comparison point
struct DenseArgs {
  const uint16_t* q;
  const uint16_t* K;
  int64_t sK_b, sK_h, sK_n;
  const uint16_t* V;
  int64_t sV_b, sV_h, sV_n;
  int B, Hq, Hkv, N;
  float sm_scale;
  float* out;
  char* ws;  // partials: B Hkv ceil(N / kSlice) (Hq / Hkv) (128 + 2) fp32
  hipStream_t stream;
};
hipError_t launch_dense(const DenseArgs& a);

hipError_t launch_select_hard(const float* err, int64_t sE_b, int64_t sE_h, int B, int Hkv, int N, int m,
                              int32_t* out, hipStream_t stream);

// Decode-time append: the cache rows the new keys and values are copied to
// (pointers already at the first new position).
struct AppendCopy {
  uint16_t* Kc;
  int64_t sKc_b, sKc_h, sKc_n;
  const uint16_t* Vn;
  int64_t sVn_b, sVn_h, sVn_n;
  uint16_t* Vc;
  int64_t sVc_b, sVc_h, sVc_n;
};

hipError_t launch_hash(const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n, int B, int Hkv,
                       int N, int L, const float* P, int64_t sP_b, int64_t sP_h, uint32_t* codes,
                       int64_t sC_b, int64_t sC_h, float* err, unsigned long long* fragile,
                       hipStream_t stream, const AppendCopy* append = nullptr);

// Algorithm 2 with the projections on the matrix cores and certified signs
// (codes and fragile count identical to launch_hash; no residual norms).
hipError_t launch_hash_mm(const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n, int B, int Hkv, int N, int L,
                          const float* P, int64_t sP_b, int64_t sP_h, uint32_t* codes, int64_t sC_b, int64_t sC_h,
                          unsigned long long* fragile, unsigned long long* fallbacks, hipStream_t stream);

hipError_t launch_build(const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n, int B, int Hkv,
                        int N, int L, const float* G, float* P, uint32_t* codes, int64_t sC_b,
                        int64_t sC_h, float* err, unsigned long long* fragile, char* ws,
                        bool checkpoint, hipStream_t stream);

// ---- device helpers ----------------------------------------------------------
__device__ __forceinline__ double bf16_to_f64(uint16_t b) {
  return (double)__uint_as_float(((uint32_t)b) << 16);
}
__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// Rounded fp64 add and multiply; the file-wide -ffp-contract=off keeps them
// from being fused.
__device__ __forceinline__ double dadd(double a, double b) { return a + b; }
__device__ __forceinline__ double dmul(double a, double b) { return a * b; }

__device__ __forceinline__ bool fragile_decision(double a) { return fabsf((float)a) < 1e-6f; }

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
// ---------------------------------------------------------------------------
// wavefront scans on DPP (no LDS round trips): within each row of 16 lanes
// by shifts of 1, 2, 4 and 8, then across rows with the broadcasts of lanes
// 15 and 31 (gfx9 DPP row_shr / row_bcast)
// ---------------------------------------------------------------------------
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ int dpp_or_zero(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, ROWS, 0xF, false);
}
// inclusive prefix sum over the 64 lanes
__device__ __forceinline__ int wave_inclusive_sum(int x) {
  x += dpp_or_zero<0x111>(x);        // row_shr:1
  x += dpp_or_zero<0x112>(x);        // row_shr:2
  x += dpp_or_zero<0x114>(x);        // row_shr:4
  x += dpp_or_zero<0x118>(x);        // row_shr:8
  x += dpp_or_zero<0x142, 0xA>(x);   // row_bcast:15 into rows 1 and 3
  x += dpp_or_zero<0x143, 0xC>(x);   // row_bcast:31 into rows 2 and 3
  return x;
}
// maximum / minimum over the 64 lanes, in every lane: quad permutations and
// row mirrors reduce each row of 16 lanes, read-lanes combine the four rows
template <bool MAX>
__device__ __forceinline__ int wave_reduce_maxmin(int x) {
  auto op = [](int a, int b) { return MAX ? max(a, b) : min(a, b); };
  x = op(x, __builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, false));   // quad_perm [1, 0, 3, 2]
  x = op(x, __builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, false));   // quad_perm [2, 3, 0, 1]
  x = op(x, __builtin_amdgcn_mov_dpp(x, 0x141, 0xF, 0xF, false));  // row_half_mirror
  x = op(x, __builtin_amdgcn_mov_dpp(x, 0x140, 0xF, 0xF, false));  // row_mirror
  return op(op(__builtin_amdgcn_readlane(x, 0), __builtin_amdgcn_readlane(x, 16)),
            op(__builtin_amdgcn_readlane(x, 32), __builtin_amdgcn_readlane(x, 48)));
}
// inclusive prefix sum within each group of 8 consecutive lanes
__device__ __forceinline__ int group8_inclusive_sum(int x) {
  const int part = threadIdx.x & 7;
  int y = dpp_or_zero<0x111>(x);
  x += (part >= 1) ? y : 0;
  y = dpp_or_zero<0x112>(x);
  x += (part >= 2) ? y : 0;
  y = dpp_or_zero<0x114>(x);
  x += (part >= 4) ? y : 0;
  return x;
}

// ---------------------------------------------------------------------------
// block-wide exclusive scan of one non-negative int per thread whose set
// bits all lie in MASK, without cross-lane shuffles: within a wavefront the
// prefix is sum_b 2^b * (lanes below with bit b set), one ballot and one
// mbcnt per bit of MASK; the wavefront totals go through LDS with one
// barrier.  Two counts can be scanned at once as (c1 << 16) | c0 when every
// sum of c0 stays below 2^16.  wave_tot[2][NW]: consecutive calls must
// alternate `buf` (0, 1, 0, ...) so that a call never overwrites totals
// another thread may still be reading.
// ---------------------------------------------------------------------------
template <int NT, uint32_t MASK>
__device__ __forceinline__ int block_exclusive_scan_bits(int v, int (*wave_tot)[NT / 64], int buf, int& total) {
  constexpr int NW = NT / 64;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  int below = 0, wtot = 0;
#pragma unroll
  for (int b = 0; b < 32; ++b) {
    if (!((MASK >> b) & 1u)) continue;
    const unsigned long long m = __ballot((v >> b) & 1);
    below += (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u)) << b;
    wtot += (int)__popcll(m) << b;
  }
  if (lane == 0) wave_tot[buf][wid] = wtot;
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int t = wave_tot[buf][w];
    before += (w < wid) ? t : 0;
    tot += t;
  }
  total = tot;
  return before + below;
}

__device__ __forceinline__ int first_lane(unsigned long long m) { return m ? __ffsll((long long)m) - 1 : 64; }

}  // namespace bpc
