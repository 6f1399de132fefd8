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
// Algorithm 1.  The fp64 residual R of every (sequence, KV head) lives in
// the workspace in dimension-major layout [bh][d][n], so that a wavefront
// whose lanes own consecutive keys reads one coalesced 512-byte line per d.
// One bit costs three launches:
//   build_dot      per key: apply the previous bit's update, store R, a = R_j . g_i,
//                  u_j = sign(a), write code bit i
//   build_reduce   per 256-key chunk: pairwise tree of u_j R_j over the chunk
//   build_finish   per (b, h): pairwise tree over chunks, v = s / N, P[i] = (float)v
// A final build_dot pass (bit == L) applies the last update and writes ||R_j||.
// The chunk trees are full binary trees over 256 rows padded with +0, so
// chunk tree + chunk-sum tree equals the pairwise tree over all N rows
// (padding only changes the sign of zero sums).
// ============================================================================

__global__ __launch_bounds__(kBuildRows) void build_dot_kernel(
    const uint16_t* __restrict__ K, int64_t sK_b, int64_t sK_h, int64_t sK_n, int Hkv, int N, int L, int bit,
    const float* __restrict__ G, const float* __restrict__ P, uint32_t* __restrict__ codes, int64_t sC_b,
    int64_t sC_h, double* __restrict__ R, float* __restrict__ err, unsigned long long* __restrict__ fragile) {
  const int bh = blockIdx.y;
  const int b = bh / Hkv, h = bh % Hkv;
  const int W = L >> 5;
  const int j = blockIdx.x * kBuildRows + threadIdx.x;
  __shared__ double g_s[kHeadDim];
  __shared__ double p_s[kHeadDim];
  __shared__ int frag_s;
  const bool final_pass = (bit == L);
  if (threadIdx.x < kHeadDim) {
    if (!final_pass) g_s[threadIdx.x] = (double)G[(size_t)bit * kHeadDim + threadIdx.x];
    if (bit > 0) p_s[threadIdx.x] = (double)P[((size_t)bh * L + (bit - 1)) * kHeadDim + threadIdx.x];
  }
  if (threadIdx.x == 0) frag_s = 0;
  __syncthreads();

  int is_fragile = 0;
  if (j < N) {
    uint32_t* crow = codes + b * sC_b + h * sC_h + (int64_t)j * W;
    bool up = false;
    if (bit > 0) up = (crow[(bit - 1) >> 5] >> ((bit - 1) & 31)) & 1u;
    double* Rj = R + (size_t)bh * kHeadDim * N + j;
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    if (bit == 0) {
      const uint16_t* krow = K + b * sK_b + h * sK_h + (int64_t)j * sK_n;
#pragma unroll
      for (int c = 0; c < kHeadDim / 8; ++c) {
        const uint4 v = *reinterpret_cast<const uint4*>(krow + 8 * c);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int d = 8 * c + e;
          const uint16_t kb = (uint16_t)((e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xFFFFu));
          const double r = bf16_to_f64(kb);
          Rj[(size_t)d * N] = r;
          acc[d >> 5] = dadd(acc[d >> 5], dmul(r, g_s[d]));
        }
      }
    } else {
#pragma unroll 8
      for (int d = 0; d < kHeadDim; ++d) {
        const double pv = p_s[d];
        double r = Rj[(size_t)d * N];
        r = r - (up ? pv : -pv);
        if (final_pass) {
          acc[d >> 5] = dadd(acc[d >> 5], dmul(r, r));
        } else {
          Rj[(size_t)d * N] = r;
          acc[d >> 5] = dadd(acc[d >> 5], dmul(r, g_s[d]));
        }
      }
    }
    const double a = dadd(dadd(acc[0], acc[1]), dadd(acc[2], acc[3]));
    if (final_pass) {
      if (err) err[(size_t)bh * N + j] = (float)sqrt(a);
    } else {
      const uint32_t ubit = (a >= 0.0) ? 1u : 0u;
      is_fragile = fragile_decision(a) ? 1 : 0;
      uint32_t* wp = crow + (bit >> 5);
      const uint32_t prev = (bit & 31) ? *wp : 0u;
      *wp = prev | (ubit << (bit & 31));
    }
  }
  if (fragile && !final_pass) {
    const unsigned long long m = __ballot(is_fragile);
    if ((threadIdx.x & 63) == 0 && m) atomicAdd(&frag_s, __popcll(m));
    __syncthreads();
    if (threadIdx.x == 0 && frag_s) atomicAdd(fragile, (unsigned long long)frag_s);
  }
}

__global__ __launch_bounds__(kBuildRows) void build_reduce_kernel(const uint32_t* __restrict__ codes,
                                                                 int64_t sC_b, int64_t sC_h, int Hkv, int N,
                                                                 int L, int bit, const double* __restrict__ R,
                                                                 double* __restrict__ part) {
  const int bh = blockIdx.y;
  const int b = bh / Hkv, h = bh % Hkv;
  const int W = L >> 5;
  const int chunk = blockIdx.x;
  const int row0 = chunk * kBuildRows;
  __shared__ double u_s[kBuildRows];
  {
    const int j = row0 + threadIdx.x;
    double u = 0.0;
    if (j < N) {
      const uint32_t w = codes[b * sC_b + h * sC_h + (int64_t)j * W + (bit >> 5)];
      u = ((w >> (bit & 31)) & 1u) ? 1.0 : -1.0;
    }
    u_s[threadIdx.x] = u;
  }
  __syncthreads();
  const int lane32 = threadIdx.x & 31;
  const int dsub = threadIdx.x >> 5;  // 0..7
  const double* Rb = R + (size_t)bh * kHeadDim * N;
  for (int dg = 0; dg < kHeadDim / 8; ++dg) {
    const int d = dg * 8 + dsub;
    const double* Rd = Rb + (size_t)d * N + row0 + lane32 * 8;
    double v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int j = row0 + lane32 * 8 + e;
      v[e] = (j < N) ? u_s[lane32 * 8 + e] * Rd[e] : 0.0;
    }
    double s = dadd(dadd(dadd(v[0], v[1]), dadd(v[2], v[3])), dadd(dadd(v[4], v[5]), dadd(v[6], v[7])));
    // pairwise across the 32 lanes of this d: partner sums are added as (mine + theirs),
    // which equals (left + right) because IEEE addition is commutative
#pragma unroll
    for (int m = 1; m < 32; m <<= 1) s = dadd(s, __shfl_xor(s, m, 64));
    if (lane32 == 0) part[((size_t)bh * gridDim.x + chunk) * kHeadDim + d] = s;
  }
}

__global__ __launch_bounds__(kHeadDim) void build_finish_kernel(int N, int L, int bit, int nchunks,
                                                               const double* __restrict__ part,
                                                               float* __restrict__ P) {
  const int bh = blockIdx.x;
  const int d = threadIdx.x;
  // pairwise tree with the odd element carried, evaluated as a binary
  // counter: a completed subtree of level l merges with the pending subtree
  // of the same level, and what remains is combined from the smallest up
  double stack_v[32];
  int stack_l[32];
  int top = 0;
  for (int c = 0; c < nchunks; ++c) {
    double x = part[((size_t)bh * nchunks + c) * kHeadDim + d];
    int lvl = 0;
    while (top > 0 && stack_l[top - 1] == lvl) {
      x = dadd(stack_v[top - 1], x);
      --top;
      ++lvl;
    }
    stack_v[top] = x;
    stack_l[top] = lvl;
    ++top;
  }
  double s = stack_v[top - 1];
  for (int t = top - 2; t >= 0; --t) s = dadd(stack_v[t], s);
  const double v = s / (double)N;
  P[((size_t)bh * L + bit) * kHeadDim + d] = (float)v;
}

hipError_t launch_build(const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n, int B, int Hkv, int N,
                        int L, const float* G, float* P, uint32_t* codes, int64_t sC_b, int64_t sC_h,
                        float* err, unsigned long long* fragile, char* ws, hipStream_t stream) {
  const BuildLayout lay = build_layout(B, Hkv, N, L);
  double* R = reinterpret_cast<double*>(ws + lay.off_R);
  double* part = reinterpret_cast<double*>(ws + lay.off_part);
  const dim3 grid(lay.nchunks, B * Hkv);
  for (int bit = 0; bit <= L; ++bit) {
    build_dot_kernel<<<grid, kBuildRows, 0, stream>>>(K, sK_b, sK_h, sK_n, Hkv, N, L, bit, G, P, codes, sC_b, sC_h,
                                                      R, err, fragile);
    if (bit == L) break;
    build_reduce_kernel<<<grid, kBuildRows, 0, stream>>>(codes, sC_b, sC_h, Hkv, N, L, bit, R, part);
    build_finish_kernel<<<B * Hkv, kHeadDim, 0, stream>>>(N, L, bit, lay.nchunks, part, P);
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
