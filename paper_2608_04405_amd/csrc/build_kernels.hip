// Prefill kernels: binary principal components (Algorithm "Constructing
// hash codes and corresponding hashing projection", Sec. 3.2) and hashing
// of keys against a given projection (Algorithm "Given projection,
// computing hashcode", Sec. 3.2).
//
// Both decide code bits from fp64 dot products in the fixed order of
// include/bpc.h, so the codes are reproducible bit for bit.

#pragma clang fp contract(off)

#include "bpc_internal.h"

namespace bpc {

// ============================================================================
// Algorithm 1.  Each bit is one pass over the keys of every (sequence, KV
// head) plus one reduction per (b, h):
//   build_bit_kernel    one workgroup per chunk of kBuildChunk keys, in groups
//                       of 64 (one key per lane); the four wavefronts of a
//                       group own the coordinate blocks [32 c, 32 c + 32), so
//                       every lane of a wavefront needs the same element of P
//                       and G at the same time and reads it as a scalar
//                       operand.  The fp64 residual of the lane's key is
//                       recomputed from the bf16 key, the key's code bits
//                       decided so far and the stored rows of P,
//                       R = (((k - u_0 P_0) - u_1 P_1) - ...), one rounded
//                       subtraction per bit (fma(-u, p, r) with u = +-1 is that
//                       subtraction: the product is exact), exactly as an
//                       in-place update would compute it.  Then a_j = R_j . g_i
//                       (fixed order), u_j and code bit i, and the chunk's
//                       pairwise tree of u_j R_j: a full binary tree over its
//                       rows, +0 past N, formed across lanes by a reduce-scatter
//                       butterfly (each level halves the coordinates a lane
//                       carries) and across the key groups in LDS.
//   build_fold_kernel   (more than 8 x 32 chunks per (b, h)) the subtrees over
//                       aligned blocks of 32 chunk sums, many workgroups
//   build_finish_kernel pairwise tree over the chunk sums (or those subtrees),
//                       v = s / N,
//                       P[i] = (float)v (and its fp64 widening for the next
//                       passes).
// A final build_bit pass (bit == L) recomputes the last residual and writes
// ||R_j||.  Without a checkpoint nothing of size N x D is stored: the pass
// reads the keys again, trading fp64 arithmetic (about L^2 D / 2 fused
// subtractions per key over the whole build) for memory traffic.  With one,
// the pass at every multiple m T of kBuildCkptPeriod also stores R after m T
// bits (1 KiB per key, in place) and the passes up to (m + 1) T start from
// it: at most T subtractions per pass, for a 1 KiB read instead of the
// 256-byte key.
// ============================================================================

// the partner lane's value at lane ^ M (quad permutes for 1 and 2)
template <int M>
__device__ __forceinline__ double xor_lane(double x) {
  if constexpr (M == 1 || M == 2) {
    constexpr int ctrl = (M == 1) ? 0xB1 : 0x4E;  // quad_perm [1,0,3,2] / [2,3,0,1]
    const int lo = __builtin_amdgcn_mov_dpp(__double2loint(x), ctrl, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_mov_dpp(__double2hiint(x), ctrl, 0xF, 0xF, false);
    return __hiloint2double(hi, lo);
  } else {
    return __shfl_xor(x, M, 64);
  }
}

// A wavefront-uniform address of data that no kernel writes while this one
// runs, in the constant address space so that loads through it are scalar.
template <typename T>
using const_ptr = const __attribute__((address_space(4))) T*;

template <typename T>
__device__ __forceinline__ const_ptr<T> uniform_ptr(const T* p) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  return (const_ptr<T>)(((uint64_t)hi << 32) | lo);
}

// one reduce-scatter level: lanes l and l ^ (1 << K) add their halves of the
// 2 * HALF coordinates they carry; the lane with bit K clear keeps the lower half
template <int K, int HALF>
__device__ __forceinline__ void rs_level(double (&v)[32], int lane) {
  const bool upper = (lane >> K) & 1;
#pragma unroll
  for (int e = 0; e < HALF; ++e) {
    const double send = upper ? v[e] : v[HALF + e];
    const double keep = upper ? v[HALF + e] : v[e];
    v[e] = dadd(keep, xor_lane<1 << K>(send));
  }
}

__global__ void build_prep_kernel(const float* __restrict__ G, double* __restrict__ G64, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) G64[i] = (double)G[i];
}

template <int W>
__global__ __launch_bounds__(kBuildThreads) void build_bit_kernel(
    const uint16_t* __restrict__ K, int64_t sK_b, int64_t sK_h, int64_t sK_n, int Hkv, int N, int L, int bit,
    const double* __restrict__ G64, const double* __restrict__ P64, uint32_t* __restrict__ codes, int64_t sC_b,
    int64_t sC_h, double* __restrict__ part, int nchunks, float* __restrict__ err,
    unsigned long long* __restrict__ fragile, double* __restrict__ ck, int ck_from, int ck_store) {
  __shared__ double xch[kBuildGroups][4][64];         // per-block partial dots of each key
  __shared__ double groot[kBuildGroups][kHeadDim];    // tree root of each key group
  __shared__ int frag;
  const int bh = blockIdx.y;
  const int b = bh / Hkv, h = bh % Hkv;
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int c = wv & 3, grp = wv >> 2;
  const bool final_pass = (bit == L);
  if (threadIdx.x == 0) frag = 0;

  const int key = blockIdx.x * kBuildChunk + grp * 64 + lane;
  const bool valid = key < N;
  double r[32];
  uint32_t cw[W];
#pragma unroll
  for (int w = 0; w < W; ++w) cw[w] = 0u;
  uint32_t* crow = codes + b * sC_b + h * sC_h + (int64_t)(valid ? key : 0) * W;
  // this lane's 32 coordinates in the checkpoint: element e of the block at
  // ckrow[(e / 2) * 64 + lane], so that each load covers 1 KiB of the
  // wavefront's keys
  typedef double f64x2 __attribute__((ext_vector_type(2)));
  f64x2* ckrow = ck ? reinterpret_cast<f64x2*>(ck + ((((size_t)bh * nchunks + blockIdx.x) * kBuildGroups + grp) * 4 +
                                                     c) * (32 * 64)) + lane
                    : nullptr;
  if (valid) {
    if (ck_from > 0) {
#pragma unroll
      for (int e2 = 0; e2 < 16; ++e2) {
        const f64x2 x = __builtin_nontemporal_load(ckrow + 64 * e2);
        r[2 * e2] = x.x;
        r[2 * e2 + 1] = x.y;
      }
    } else {
      const uint16_t* krow = K + b * sK_b + h * sK_h + (int64_t)key * sK_n + 32 * c;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint4 v = *reinterpret_cast<const uint4*>(krow + 8 * q);
        const uint32_t wd[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 8; ++e)
          r[8 * q + e] = bf16_to_f64((uint16_t)((e & 1) ? (wd[e >> 1] >> 16) : (wd[e >> 1] & 0xFFFFu)));
      }
    }
#pragma unroll
    for (int w = 0; w < W; ++w)
      if (32 * w < bit) cw[w] = crow[w];
  } else {
#pragma unroll
    for (int e = 0; e < 32; ++e) r[e] = 0.0;  // never contributes: padded below
  }
  // the residual after bits 0 .. bit - 1: bits ck_from .. bit - 1 removed
  // from the checkpoint (or all of them from the key)
  const_ptr<double> prow = uniform_ptr(P64 + (size_t)bh * L * kHeadDim + 32 * c);
#pragma unroll
  for (int w = 0; w < W; ++w) {
    const int ib0 = max(0, ck_from - 32 * w);
    const int nb = min(32, bit - 32 * w);
    const uint32_t word = cw[w];
    for (int ib = ib0; ib < nb; ++ib) {
      const double sg = ((word >> ib) & 1u) ? -1.0 : 1.0;
      const_ptr<double> p = prow + (size_t)(32 * w + ib) * kHeadDim;
#pragma unroll
      for (int e = 0; e < 32; ++e) r[e] = __builtin_fma(sg, p[e], r[e]);
    }
  }
  if (ck_store && valid) {
#pragma unroll
    for (int e2 = 0; e2 < 16; ++e2) {
      const f64x2 x = {r[2 * e2], r[2 * e2 + 1]};
      __builtin_nontemporal_store(x, ckrow + 64 * e2);
    }
  }
  if (final_pass) {
    double sq = 0.0;
#pragma unroll
    for (int e = 0; e < 32; ++e) sq = dadd(sq, dmul(r[e], r[e]));
    xch[grp][c][lane] = sq;
    __syncthreads();
    if (err && c == 0 && valid)
      err[(size_t)bh * N + key] = (float)sqrt(dadd(dadd(xch[grp][0][lane], xch[grp][1][lane]),
                                                   dadd(xch[grp][2][lane], xch[grp][3][lane])));
    return;
  }
  // a_j = R_j . g (four blocks of 32, ascending, combined ((b0 + b1) + (b2 + b3)))
  const_ptr<double> g = uniform_ptr(G64 + (size_t)bit * kHeadDim + 32 * c);
  double acc = 0.0;
#pragma unroll
  for (int e = 0; e < 32; ++e) acc = dadd(acc, dmul(r[e], g[e]));
  xch[grp][c][lane] = acc;
  __syncthreads();
  const double a =
      dadd(dadd(xch[grp][0][lane], xch[grp][1][lane]), dadd(xch[grp][2][lane], xch[grp][3][lane]));
  const bool u = a >= 0.0;
  if (c == 0) {
    if (valid) crow[bit >> 5] = ((bit & 31) ? cw[bit >> 5] : 0u) | ((u ? 1u : 0u) << (bit & 31));
    if (fragile) {
      const unsigned long long m = __ballot(valid && fragile_decision(a));
      if (lane == 0 && m) atomicAdd(&frag, __popcll(m));
    }
  }
  // u_j R_j (exact), keys past N padded with +0, and the tree over the
  // group's 64 keys: after the five reduce-scatter levels lane l carries the
  // coordinate whose index is l's low five bits reversed, summed over its
  // half of the group; the xor-32 step adds the two halves
  double v[32];
#pragma unroll
  for (int e = 0; e < 32; ++e) v[e] = valid ? (u ? r[e] : -r[e]) : 0.0;
  rs_level<0, 16>(v, lane);
  rs_level<1, 8>(v, lane);
  rs_level<2, 4>(v, lane);
  rs_level<3, 2>(v, lane);
  rs_level<4, 1>(v, lane);
  const double s = dadd(v[0], xor_lane<32>(v[0]));
  if (lane < 32) {
    const int e = (int)(__brev((uint32_t)lane) >> 27);
    groot[grp][32 * c + e] = s;
  }
  __syncthreads();
  static_assert(kBuildGroups == 2, "one tree level across the key groups");
  if (threadIdx.x < kHeadDim)
    part[((size_t)bh * nchunks + blockIdx.x) * kHeadDim + threadIdx.x] =
        dadd(groot[0][threadIdx.x], groot[1][threadIdx.x]);
  if (fragile && threadIdx.x == 0 && frag) atomicAdd(fragile, (unsigned long long)frag);
}

// Thread d of workgroup (x, bh) folds the aligned block of chunk sums
// [x kBuildFold, (x + 1) kBuildFold) of coordinate d, level by level with the
// odd one carried (the last block may be short): the subtree of the pairwise
// tree over those chunks.
__global__ __launch_bounds__(kHeadDim) void build_fold_kernel(const double* __restrict__ part, int nchunks,
                                                              double* __restrict__ fold, int nfold) {
  const int bh = blockIdx.y, x = blockIdx.x, d = threadIdx.x;
  const int begin = x * kBuildFold;
  int c = min(kBuildFold, nchunks - begin);
  const double* src = part + ((size_t)bh * nchunks + begin) * kHeadDim + d;
  double v[kBuildFold];
#pragma unroll
  for (int e = 0; e < kBuildFold; ++e) v[e] = (e < c) ? src[(size_t)e * kHeadDim] : 0.0;
#pragma unroll
  for (int w = kBuildFold / 2; w >= 1; w >>= 1) {
#pragma unroll
    for (int i = 0; i < w; ++i) v[i] = (2 * i + 1 < c) ? dadd(v[2 * i], v[2 * i + 1]) : v[2 * i];
    c = (c + 1) >> 1;
  }
  fold[((size_t)bh * nfold + x) * kHeadDim + d] = v[0];
}

// One workgroup per (b, h): thread (blk, d) folds an aligned block of S
// chunk sums of coordinate d (S a power of two, 8 blocks cover all chunks) as
// a binary counter, and the block roots are then paired level by level in LDS
// with the odd one carried.  Both are the pairwise tree with the odd element
// carried: a binary counter's final right fold equals level-wise pairing, and
// level-wise pairing of the leaves splits at every aligned power of two.
constexpr int kFinishBlocks = 8;

__global__ __launch_bounds__(kFinishBlocks* kHeadDim) void build_finish_kernel(int N, int L, int bit, int nchunks,
                                                                               const double* __restrict__ part,
                                                                               float* __restrict__ P,
                                                                               double* __restrict__ P64) {
  __shared__ double node[kFinishBlocks][kHeadDim];
  const int bh = blockIdx.x;
  const int d = threadIdx.x & (kHeadDim - 1), blk = threadIdx.x >> 7;
  int S = 1;
  while (S * kFinishBlocks < nchunks) S <<= 1;
  const int begin = blk * S, end = min(begin + S, nchunks);
  const double* src = part + (size_t)bh * nchunks * kHeadDim + d;
  double stack_v[32];
  int stack_l[32];
  int top = 0;
  for (int c0 = begin; c0 < end; c0 += 8) {
    double x[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = (c0 + e < end) ? src[(size_t)(c0 + e) * kHeadDim] : 0.0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (c0 + e >= end) break;
      double y = x[e];
      int lvl = 0;
      while (top > 0 && stack_l[top - 1] == lvl) {
        y = dadd(stack_v[top - 1], y);
        --top;
        ++lvl;
      }
      stack_v[top] = y;
      stack_l[top] = lvl;
      ++top;
    }
  }
  if (top > 0) {
    double y = stack_v[top - 1];
    for (int t = top - 2; t >= 0; --t) y = dadd(stack_v[t], y);
    node[blk][d] = y;
  }
  int cnt = (nchunks + S - 1) / S;
  while (cnt > 1) {
    __syncthreads();
    const int half = (cnt + 1) >> 1;
    double y = 0.0;
    if (blk < half) y = (2 * blk + 1 < cnt) ? dadd(node[2 * blk][d], node[2 * blk + 1][d]) : node[2 * blk][d];
    __syncthreads();
    if (blk < half) node[blk][d] = y;
    cnt = half;
  }
  if (blk == 0) {
    const double v = node[0][d] / (double)N;
    const float pf = (float)v;
    P[((size_t)bh * L + bit) * kHeadDim + d] = pf;
    P64[((size_t)bh * L + bit) * kHeadDim + d] = (double)pf;
  }
}

template <int W>
static void launch_build_W(const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n, int B, int Hkv, int N,
                           int L, const double* G64, float* P, double* P64, uint32_t* codes, int64_t sC_b,
                           int64_t sC_h, float* err, unsigned long long* fragile, double* part, int nchunks,
                           double* fold, int nfold, double* ck, hipStream_t stream) {
  const dim3 grid(nchunks, B * Hkv);
  for (int bit = 0; bit <= L; ++bit) {
    // With a checkpoint buffer the pass at bit m T stores R after m T bits,
    // and the passes up to the next one start from it.
    int from = 0, store = 0;
    if (ck) {
      from = bit - (bit % kBuildCkptPeriod == 0 ? kBuildCkptPeriod : bit % kBuildCkptPeriod);
      from = max(from, 0);
      store = (bit > 0 && bit < L && bit % kBuildCkptPeriod == 0) ? 1 : 0;
    }
    build_bit_kernel<W><<<grid, kBuildThreads, 0, stream>>>(K, sK_b, sK_h, sK_n, Hkv, N, L, bit, G64, P64, codes,
                                                           sC_b, sC_h, part, nchunks, err, fragile, ck, from,
                                                           store);
    if (bit == L) break;
    if (nfold) {
      build_fold_kernel<<<dim3(nfold, B * Hkv), kHeadDim, 0, stream>>>(part, nchunks, fold, nfold);
      build_finish_kernel<<<B * Hkv, kFinishBlocks * kHeadDim, 0, stream>>>(N, L, bit, nfold, fold, P, P64);
    } else {
      build_finish_kernel<<<B * Hkv, kFinishBlocks * kHeadDim, 0, stream>>>(N, L, bit, nchunks, part, P, P64);
    }
  }
}

hipError_t launch_build(const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n, int B, int Hkv, int N,
                        int L, const float* G, float* P, uint32_t* codes, int64_t sC_b, int64_t sC_h,
                        float* err, unsigned long long* fragile, char* ws, bool checkpoint, hipStream_t stream) {
  const BuildLayout lay = build_layout(B, Hkv, N, L);
  double* part = reinterpret_cast<double*>(ws + lay.off_part);
  double* ck = checkpoint ? reinterpret_cast<double*>(ws + lay.off_ck) : nullptr;
  double* fold = reinterpret_cast<double*>(ws + lay.off_fold);
  double* P64 = reinterpret_cast<double*>(ws + lay.off_p64);
  double* G64 = reinterpret_cast<double*>(ws + lay.off_g64);
  const int ng = L * kHeadDim;
  build_prep_kernel<<<(ng + 255) / 256, 256, 0, stream>>>(G, G64, ng);
  switch (L) {
    case 32:
      launch_build_W<1>(K, sK_b, sK_h, sK_n, B, Hkv, N, L, G64, P, P64, codes, sC_b, sC_h, err, fragile, part,
                        lay.nchunks, fold, lay.nfold, ck, stream);
      break;
    case 64:
      launch_build_W<2>(K, sK_b, sK_h, sK_n, B, Hkv, N, L, G64, P, P64, codes, sC_b, sC_h, err, fragile, part,
                        lay.nchunks, fold, lay.nfold, ck, stream);
      break;
    default:
      launch_build_W<4>(K, sK_b, sK_h, sK_n, B, Hkv, N, L, G64, P, P64, codes, sC_b, sC_h, err, fragile, part,
                        lay.nchunks, fold, lay.nfold, ck, stream);
      break;
  }
  return hipGetLastError();
}

// ============================================================================
// Algorithm 2.  Four lanes per key: lane q of a quad holds the fp64
// residual of coordinates [32q, 32q + 32) in registers, so each bit's dot
// product is four sequential block sums combined across the quad as
// ((b0 + b1) + (b2 + b3)) -- the fixed order -- and the residual update
// needs no communication.  The projection is staged in LDS once per
// workgroup (padded rows avoid bank conflicts between the four blocks).
// ============================================================================

// With a cache copy (cp.Kc non-null), decode-time append: each key row of K
// (the new keys) is also stored into the cache rows cp.Kc, and the matching
// value rows cp.Vn into cp.Vc; the four lanes of a key each move a quarter
// of both rows.
template <int L>
__global__ __launch_bounds__(256) void hash_kernel(const uint16_t* __restrict__ K, int64_t sK_b, int64_t sK_h,
                                                   int64_t sK_n, int Hkv, int N, const float* __restrict__ P,
                                                   int64_t sP_b, int64_t sP_h, uint32_t* __restrict__ codes,
                                                   int64_t sC_b, int64_t sC_h, float* __restrict__ err,
                                                   unsigned long long* __restrict__ fragile, AppendCopy cp) {
  constexpr int W = L / 32;
  constexpr int PAD = 33;
  __shared__ float p_s[L][4][PAD];
  __shared__ int frag_s;
  const int bh = blockIdx.y;
  const int b = bh / Hkv, h = bh % Hkv;
  const float* Pb = P + b * sP_b + h * sP_h;
  for (int e = threadIdx.x; e < L * kHeadDim; e += 256) {
    const int i = e / kHeadDim, d = e % kHeadDim;
    p_s[i][d >> 5][d & 31] = Pb[e];
  }
  if (threadIdx.x == 0) frag_s = 0;
  __syncthreads();

  const int key = blockIdx.x * 64 + (threadIdx.x >> 2);
  const int qd = threadIdx.x & 3;
  const bool valid = key < N;
  double r[32];
  if (valid) {
    const uint16_t* krow = K + b * sK_b + h * sK_h + (int64_t)key * sK_n + 32 * qd;
    uint4 kq[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const uint4 v = *reinterpret_cast<const uint4*>(krow + 8 * c);
      kq[c] = v;
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 8; ++e)
        r[8 * c + e] = bf16_to_f64((uint16_t)((e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xFFFFu)));
    }
    if (cp.Kc) {
      uint16_t* kc = cp.Kc + b * cp.sKc_b + h * cp.sKc_h + (int64_t)key * cp.sKc_n + 32 * qd;
      const uint16_t* vn = cp.Vn + b * cp.sVn_b + h * cp.sVn_h + (int64_t)key * cp.sVn_n + 32 * qd;
      uint16_t* vc = cp.Vc + b * cp.sVc_b + h * cp.sVc_h + (int64_t)key * cp.sVc_n + 32 * qd;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        reinterpret_cast<uint4*>(kc)[c] = kq[c];
        reinterpret_cast<uint4*>(vc)[c] = reinterpret_cast<const uint4*>(vn)[c];
      }
    }
  } else {
#pragma unroll
    for (int e = 0; e < 32; ++e) r[e] = 0.0;
  }
  uint32_t word = 0;
  int nfrag = 0;
  for (int i = 0; i < L; ++i) {
    double acc = 0.0;
#pragma unroll
    for (int e = 0; e < 32; ++e) acc = dadd(acc, dmul(r[e], (double)p_s[i][qd][e]));
    const double s01 = dadd(acc, __shfl_xor(acc, 1, 64));
    const double a = dadd(s01, __shfl_xor(s01, 2, 64));
    const bool u = a >= 0.0;
    if (qd == 0 && valid && fragile_decision(a)) ++nfrag;
    if ((i >> 5) == qd && u) word |= 1u << (i & 31);
#pragma unroll
    for (int e = 0; e < 32; ++e) {
      const double pv = (double)p_s[i][qd][e];
      r[e] = r[e] - (u ? pv : -pv);
    }
  }
  if (valid && qd < W) codes[b * sC_b + h * sC_h + (int64_t)key * W + qd] = word;
  if (err) {
    double sq = 0.0;
#pragma unroll
    for (int e = 0; e < 32; ++e) sq = dadd(sq, dmul(r[e], r[e]));
    const double s01 = dadd(sq, __shfl_xor(sq, 1, 64));
    const double tot = dadd(s01, __shfl_xor(s01, 2, 64));
    if (valid && qd == 0) err[(size_t)bh * N + key] = (float)sqrt(tot);
  }
  if (fragile) {
    int wsum = nfrag;
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) wsum += __shfl_xor(wsum, m, 64);
    if ((threadIdx.x & 63) == 0 && wsum) atomicAdd(&frag_s, wsum);
    __syncthreads();
    if (threadIdx.x == 0 && frag_s) atomicAdd(fragile, (unsigned long long)frag_s);
  }
}

hipError_t launch_hash(const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n, int B, int Hkv, int N, int L,
                       const float* P, int64_t sP_b, int64_t sP_h, uint32_t* codes, int64_t sC_b, int64_t sC_h,
                       float* err, unsigned long long* fragile, hipStream_t stream, const AppendCopy* append) {
  const dim3 grid((N + 63) / 64, B * Hkv);
  const AppendCopy cp = append ? *append : AppendCopy{};
  switch (L) {
    case 32:
      hash_kernel<32><<<grid, 256, 0, stream>>>(K, sK_b, sK_h, sK_n, Hkv, N, P, sP_b, sP_h, codes, sC_b, sC_h, err,
                                                fragile, cp);
      break;
    case 64:
      hash_kernel<64><<<grid, 256, 0, stream>>>(K, sK_b, sK_h, sK_n, Hkv, N, P, sP_b, sP_h, codes, sC_b, sC_h, err,
                                                fragile, cp);
      break;
    default:
      hash_kernel<128><<<grid, 256, 0, stream>>>(K, sK_b, sK_h, sK_n, Hkv, N, P, sP_b, sP_h, codes, sC_b, sC_h,
                                                 err, fragile, cp);
      break;
  }
  return hipGetLastError();
}

}  // namespace bpc
