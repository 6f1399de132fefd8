// Algorithm 2 ("Given projection, computing hashcode"; App A.3, hashing
// kernel) with the projections on the matrix cores and every sign certified
// against the fixed-order fp64 arithmetic of bpc_hash_keys.
//
// The iterative residual r_{i+1} = r_i - u_i P_i makes bit i depend on the
// signs before it only through the Gram matrix of P:
//
//     a_i = r_i . P_i = k . P_i - sum_{t<i} u_t (P_t . P_i),
//
// so the N x L products k . P_i are one dense contraction (K times P^T), and
// what stays sequential per key is an L x L triangle of corrections.  The
// contraction runs as bf16 MFMA: a bf16 key times fp32 P is exact once P is
// cut into three bf16 parts (hi + mid + lo, by truncation, exactly P), and
// the products accumulate in fp32.  The corrections run in fp32 on the
// vector units with the Gram matrix (fp64, rounded to fp32) as wavefront-
// uniform operands; at L >= 64 the corrections by earlier 16-bit blocks are
// one more bf16 contraction (signs +-1 times the Gram entries cut like P,
// the hi products in a chain of their own) and only each block's own
// triangle stays on the vector units.
//
// The fp32 value a^ differs from the value a the fixed-order fp64 reference
// computes (canonical residual, four-block dot) by at most
//
//   E_i = 136 u S + (i + 2) u (|a^| + 2.01 C_i) + (36 + i) 2^-53 (S + Q_i)
//         + |k| 2^-100 + 2^-110,                     u = 2^-24,
//
// S = |k| |P_i| >= sum_d |k_d P_id| (Cauchy-Schwarz), C_i = sum_{t<i}
// |P_t . P_i| (inflated for the Gram matrix's own fp64 error), Q_i =
// sum_d (sum_t |P_td|) |P_id|.  The first term is fp32 accumulation inside
// the MFMA chains (each of the four 32-coordinate hi-part steps adds at most
// 32 roundings of the running sum; the mid and lo parts, 2^-8 and 2^-16 of
// the size, are accumulated apart and added once), the second the
// corrections and the Gram matrix's rounding to fp32, the third the
// reference's own rounding (i rounded subtractions per coordinate and the
// 34 roundings of a four-block dot), the last two underflow of bf16 parts
// and products.  With the corrections on the matrix cores the bound takes
// 138 u S, (i + 4) in place of (i + 2) before 2.01 C_i, and 2^-109: the
// mid/lo chain gains at most 32 roundings per earlier block of sums below
// 2^-7 (S + C_i), the hi chain at most 16 T roundings of sums below C_i, and
// one addition joins it.  The evaluation of E_i in fp32 is covered by a factor
// 1 + 2^-8.  When |a^| > E_i + 1.01e-6 the reference's sign is that of a^,
// and |fp32(a)| >= 1e-6, so the decision is not fragile.  Otherwise (a few
// keys in ten thousand, and every decision near zero), the wavefront
// recomputes that one decision in the reference arithmetic: the residual
// rebuilt from the bf16 key with one rounded subtraction per earlier bit, in
// order, and the four-block dot; the fragile test is then the reference's.
// Non-finite values make every comparison fail and take the same route.

#include "bpc_internal.h"

namespace bpc {

typedef short bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// 64 keys per wavefront per iteration; four wavefronts per workgroup, eight
// at L = 128, where one workgroup fills a CU's LDS
template <int L>
constexpr int hm_threads() { return L == 128 ? 512 : 256; }
constexpr int kHmPsStride = 132;     // fp32 P row stride in LDS (floats)
constexpr int kHmXsStride = 20;      // transpose buffer row stride (floats)

// D += A B for one 16 x 16 x 32 bf16 tile (fp32 accumulation).  Lane i
// supplies A[i % 16][8 (i / 16) + j] and B[8 (i / 16) + j][i % 16] for
// j = 0..7 (two bf16 per word, low half first) and holds D[4 (i / 16) + j]
// [i % 16] for j = 0..3.  The order of the coordinates inside a lane only has
// to agree between A and B.
__device__ __forceinline__ f32x4_t mfma32(const uint4 a, const uint4 b, f32x4_t d) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                 d, 0, 0, 0);
}

// Eight fp32 values cut exactly into three bf16 parts: hi keeps the top 8
// significant bits, mid the next 8, lo the rest (at most 8 significant bits
// remain once hi and mid are subtracted; both subtractions are exact).
__device__ __forceinline__ void split3(const float4 p0, const float4 p1, uint4& hi, uint4& mid, uint4& lo) {
  const float v[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
  uint32_t h[8], m[8], l[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t bh = __float_as_uint(v[e]) & 0xFFFF0000u;
    const float r1 = v[e] - __uint_as_float(bh);
    const uint32_t bm = __float_as_uint(r1) & 0xFFFF0000u;
    const float r2 = r1 - __uint_as_float(bm);
    h[e] = bh, m[e] = bm, l[e] = __float_as_uint(r2);
  }
  hi = make_uint4(__builtin_amdgcn_perm(h[1], h[0], 0x07060302u), __builtin_amdgcn_perm(h[3], h[2], 0x07060302u),
                  __builtin_amdgcn_perm(h[5], h[4], 0x07060302u), __builtin_amdgcn_perm(h[7], h[6], 0x07060302u));
  mid = make_uint4(__builtin_amdgcn_perm(m[1], m[0], 0x07060302u), __builtin_amdgcn_perm(m[3], m[2], 0x07060302u),
                   __builtin_amdgcn_perm(m[5], m[4], 0x07060302u), __builtin_amdgcn_perm(m[7], m[6], 0x07060302u));
  lo = make_uint4(__builtin_amdgcn_perm(l[1], l[0], 0x07060302u), __builtin_amdgcn_perm(l[3], l[2], 0x07060302u),
                  __builtin_amdgcn_perm(l[5], l[4], 0x07060302u), __builtin_amdgcn_perm(l[7], l[6], 0x07060302u));
}

__device__ __forceinline__ void wave_lds_sync() {
  // LDS operations of one wavefront complete in order; the fences keep the
  // compiler from moving LDS accesses across this point
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ double readlane_f64(double x, int lane) {
  const uint64_t b = __double_as_longlong(x);
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)b, lane);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(b >> 32), lane);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}


// Decision `bit` of one key in the reference arithmetic, computed by the
// whole wavefront: lane l carries coordinates l and l + 64 of the residual,
// rebuilt from the bf16 key with one rounded subtraction per earlier bit in
// ascending order; the products are rounded, then each block of 32
// coordinates is summed in ascending order from +0 and the blocks combined
// as ((b0 + b1) + (b2 + b3)).  krow and u0..u3 (the key's code words so far)
// are the same in every lane; fb is the wavefront's scratch of 128 doubles.
__device__ __forceinline__ double hm_reference_decision(const uint16_t* krow, const float* Ps, int bit, uint32_t u0,
                                                     uint32_t u1, uint32_t u2, uint32_t u3, double* fb) {
  const int l = threadIdx.x & 63;
  double r0 = bf16_to_f64(krow[l]), r1 = bf16_to_f64(krow[l + 64]);
  for (int t = 0; t < bit; ++t) {
    const int q = t >> 5;
    const uint32_t word = q == 0 ? u0 : q == 1 ? u1 : q == 2 ? u2 : u3;
    const bool ut = (word >> (t & 31)) & 1u;
    const double p0 = (double)Ps[t * kHmPsStride + l], p1 = (double)Ps[t * kHmPsStride + l + 64];
    r0 = ut ? r0 - p0 : r0 + p0;
    r1 = ut ? r1 - p1 : r1 + p1;
  }
  fb[l] = dmul(r0, (double)Ps[bit * kHmPsStride + l]);
  fb[64 + l] = dmul(r1, (double)Ps[bit * kHmPsStride + l + 64]);
  wave_lds_sync();
  double s = 0.0;
  if (l < 4) {
#pragma unroll 8
    for (int e = 0; e < 32; ++e) s = dadd(s, fb[32 * l + e]);
  }
  const double s0 = readlane_f64(s, 0), s1 = readlane_f64(s, 1), s2 = readlane_f64(s, 2), s3 = readlane_f64(s, 3);
  wave_lds_sync();  // fb is rewritten by the next call only after these reads
  return dadd(dadd(s0, s1), dadd(s2, s3));
}

// The Gram matrix by rows, each row t holding the 16-wide column blocks from
// t's own block on: G[t][i] (t < i) at hm_gram_row<L>(t) + i - 16 (t / 16).
template <int L>
__device__ __forceinline__ int hm_gram_row(int t) {
  constexpr int nb = L / 16;
  const int a = t >> 4, r = t & 15;
  return 16 * (16 * (nb * a - a * (a - 1) / 2) + r * (nb - a));
}
template <int L>
constexpr int hm_gram_size() { return 256 * (L / 16) * (L / 16 + 1) / 2; }

// At L >= 64 the corrections by earlier blocks run on the matrix cores (see
// the main loop), and the Gram matrix (the same size) is kept as the 16 x 16
// diagonal blocks (row t, column i % 16 at 256 (t / 16) + 16 (t % 16) +
// i % 16), then, for every bit i of block T >= 1, the 16 T entries G[t][i],
// t < 16 T, contiguous (the matrix-core operand reads 8 consecutive t).
template <int L>
constexpr bool hm_mm_corr() { return L >= 64; }
template <int L>
__device__ __forceinline__ int hm_gram_col(int i) {  // the entries G[t][i], t < 16 (i / 16)
  constexpr int nb = L / 16;
  const int T = i >> 4;
  return 256 * nb + 256 * (T * (T - 1) / 2) + 16 * T * (i & 15);
}
// the index of G[t][i], t < i
template <int L>
__device__ __forceinline__ int hm_gram_at(int t, int i) {
  if constexpr (hm_mm_corr<L>()) {
    if ((t >> 4) == (i >> 4)) return 256 * (t >> 4) + 16 * (t & 15) + (i & 15);
    return hm_gram_col<L>(i) + t;
  } else {
    return hm_gram_row<L>(t) + i - 16 * (t >> 4);
  }
}
// G[t][16 (t / 16) .. + 15], the row of t inside its own column block
template <int L>
__device__ __forceinline__ int hm_gram_diag(int t) {
  if constexpr (hm_mm_corr<L>()) return 256 * (t >> 4) + 16 * (t & 15);
  else return hm_gram_row<L>(t);
}

// Eight bf16 operands +-1 from the bits of `byte` (bit set: -1), low half of
// each word first; all zero when !on
__device__ __forceinline__ uint4 sign_operand(uint32_t byte, bool on) {
  uint32_t w[4];
#pragma unroll
  for (int k = 0; k < 4; ++k)
    w[k] = on ? (0x3F803F80u | (((byte >> (2 * k)) & 1u) << 15) | (((byte >> (2 * k + 1)) & 1u) << 31)) : 0u;
  return make_uint4(w[0], w[1], w[2], w[3]);
}

template <int L>
struct HmShared {
  float Ps[L * kHmPsStride];              // P of this (b, h), fp32
  float Gs[hm_gram_size<L>()];            // fp32(P_t . P_i) for t < i, at hm_gram_at(t, i)
  float4 cst[L];                          // per bit: |P_i|, c1, c2, c3 (see hm_bound)
  float Xs[hm_threads<L>() / 64][64 * kHmXsStride];  // per wavefront: MFMA tile -> one key per lane (also setup scratch)
  unsigned int nfrag, nfall;
};

template <int L>
__global__ __launch_bounds__(hm_threads<L>(), 2) void hash_mm_kernel(const uint16_t* __restrict__ K, int64_t sK_b,
                                                             int64_t sK_h, int64_t sK_n, int Hkv, int N,
                                                             const float* __restrict__ P, int64_t sP_b, int64_t sP_h,
                                                             uint32_t* __restrict__ codes, int64_t sC_b,
                                                             int64_t sC_h, unsigned long long* __restrict__ fragile,
                                                             unsigned long long* __restrict__ fallbacks,
                                                             int keys_per_wg) {
  constexpr int W = L / 32;
  constexpr int kHmThreads = hm_threads<L>();
  constexpr int NWV = kHmThreads / 64;
  __shared__ __align__(16) HmShared<L> sh;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int bh = blockIdx.y;
  const int b = bh / Hkv, h = bh % Hkv;
  const float* Pb = P + b * sP_b + h * sP_h;
  const uint16_t* Kb = K + b * sK_b + h * sK_h;

  // ---- set-up: P, its Gram matrix and the per-bit bound constants ----------
  for (int e = tid; e < L * 32; e += kHmThreads) {
    const int i = e >> 5, c = e & 31;
    *reinterpret_cast<float4*>(&sh.Ps[i * kHmPsStride + 4 * c]) = reinterpret_cast<const float4*>(Pb)[e];
  }
  if (tid == 0) sh.nfrag = 0, sh.nfall = 0;
  __syncthreads();
  double* Ad = reinterpret_cast<double*>(&sh.Xs[0][0]);  // sum_t |P_td|, [128]
  double* nP = Ad + kHeadDim;                             // |P_t| in fp64, [L]
  for (int e = tid; e < L * L; e += kHmThreads) {
    const int t = e / L, i = e % L;
    if (t < i) {
      double s = 0.0;
      for (int d = 0; d < kHeadDim; d += 4) {
        const float4 x = *reinterpret_cast<const float4*>(&sh.Ps[t * kHmPsStride + d]);
        const float4 y = *reinterpret_cast<const float4*>(&sh.Ps[i * kHmPsStride + d]);
        s = fma((double)x.x, (double)y.x, s);
        s = fma((double)x.y, (double)y.y, s);
        s = fma((double)x.z, (double)y.z, s);
        s = fma((double)x.w, (double)y.w, s);
      }
      sh.Gs[hm_gram_at<L>(t, i)] = (float)s;
    }
  }
  if (tid < kHeadDim) {
    double a = 0.0;
    for (int t = 0; t < L; ++t) a += fabs((double)sh.Ps[t * kHmPsStride + tid]);
    Ad[tid] = a;
  } else if (tid - kHeadDim < L) {
    const int t = tid - kHeadDim;
    double s = 0.0;
    for (int d = 0; d < kHeadDim; ++d) s = fma((double)sh.Ps[t * kHmPsStride + d], (double)sh.Ps[t * kHmPsStride + d], s);
    nP[t] = sqrt(s) * (1.0 + 0x1p-40);
  }
  __syncthreads();
  if (tid < L) {
    const int i = tid;
    double cabs = 0.0, q = 0.0;
    for (int t = 0; t < i; ++t)
      cabs += fabs((double)sh.Gs[hm_gram_at<L>(t, i)]) + 0x1p-20 * nP[t] * nP[i];
    for (int d = 0; d < kHeadDim; ++d) q += Ad[d] * fabs((double)sh.Ps[i * kHmPsStride + d]);
    const double up = 1.0 + 0x1p-20;
    // with the corrections on the matrix cores: two more roundings of
    // 2^-7-sized sums per earlier bit in the mid/lo chain (+2 u S, +2 u C_i)
    constexpr bool mm = hm_mm_corr<L>();
    const double c1 = ((mm ? 138.0 : 136.0) * 0x1p-24 + (36.0 + i) * 0x1p-53) * up;
    const double c2 = (i + 2.0) * 0x1p-24;
    const double c3 = ((i + (mm ? 4.0 : 2.0)) * 0x1p-24 * 2.01 * cabs + q * (36.0 + i) * 0x1p-53 +
                       (mm ? 0x1p-109 : 0x1p-110) + 1.01e-6) *
                      up;
    sh.cst[i] = make_float4((float)(nP[i] * up) * (float)up, (float)c1, (float)c2, (float)c3);
  }
  __syncthreads();

  // ---- main loop: 64 keys per wavefront per iteration --------------------
  const int c16 = lane & 15, g4 = lane >> 4;
  float* Xs = sh.Xs[wave];
  double* fb = reinterpret_cast<double*>(Xs);
  const int key_begin = blockIdx.x * keys_per_wg;
  const int key_end = min(N, key_begin + keys_per_wg);
  unsigned int nfrag = 0, nfall = 0;
  for (int base = key_begin + wave * 64; base < key_end; base += NWV * 64) {
    // B operands: lane i holds key base + 16 tau + i % 16, coordinates
    // 32 m + 8 (i / 16) .. + 7
    uint4 kv[4][4];
    float ss[4];
#pragma unroll
    for (int tau = 0; tau < 4; ++tau) {
      const int key = base + 16 * tau + c16;
      ss[tau] = 0.f;
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        kv[tau][m] = key < key_end ? *reinterpret_cast<const uint4*>(Kb + (int64_t)key * sK_n + 32 * m + 8 * g4)
                                   : make_uint4(0u, 0u, 0u, 0u);
        const uint32_t wv[4] = {kv[tau][m].x, kv[tau][m].y, kv[tau][m].z, kv[tau][m].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lo = bf16_to_f32(wv[e] & 0xFFFFu), hi = bf16_to_f32(wv[e] >> 16);
          ss[tau] = fmaf(lo, lo, ss[tau]);
          ss[tau] = fmaf(hi, hi, ss[tau]);
        }
      }
      ss[tau] += __shfl_xor(ss[tau], 16, 64);
      ss[tau] += __shfl_xor(ss[tau], 32, 64);
    }
    // from here on lane l owns key base + l (its norm sits in ss[l / 16])
    const float ssq = g4 == 0 ? ss[0] : g4 == 1 ? ss[1] : g4 == 2 ? ss[2] : ss[3];
    const float nk = sqrtf(ssq * (1.f + 0x1p-14f)) * (1.f + 0x1p-20f);
    const float nkx = nk * 0x1p-100f;
    const bool valid = base + lane < key_end;
    const uint16_t* my_row = Kb + (int64_t)(base + lane) * sK_n;
    uint32_t cw[W];
#pragma unroll
    for (int w = 0; w < W; ++w) cw[w] = 0u;

#pragma unroll
    for (int T = 0; T < L / 16; ++T) {
      // projections of bits 16 T .. 16 T + 15 of the 64 keys
      f32x4_t ah[4], as[4], ch[4];
#pragma unroll
      for (int tau = 0; tau < 4; ++tau) ah[tau] = as[tau] = ch[tau] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const float* prow = &sh.Ps[(16 * T + c16) * kHmPsStride + 32 * m + 8 * g4];
        uint4 phi, pmid, plo;
        split3(*reinterpret_cast<const float4*>(prow), *reinterpret_cast<const float4*>(prow + 4), phi, pmid, plo);
#pragma unroll
        for (int tau = 0; tau < 4; ++tau) {
          as[tau] = mfma32(plo, kv[tau][m], as[tau]);
          as[tau] = mfma32(pmid, kv[tau][m], as[tau]);
          ah[tau] = mfma32(phi, kv[tau][m], ah[tau]);
        }
      }
      if constexpr (hm_mm_corr<L>()) {
        // The corrections by earlier blocks as one more contraction: D[j][key]
        // = sum_{t < 16 T} fp32(G[t][16 T + j]) s_t(key), s_t = -1 where bit t
        // of the key is set, else +1 (exact in bf16).  Gram entries are cut
        // into hi + mid + lo like P; the hi products go to their own chain
        // ch (sums of size C_i), mid and lo to the small chain as.
#pragma unroll
        for (int st = 0; st < (T + 1) / 2; ++st) {
          const uint32_t cws = cw[st];
          // lane (g4, c16): A = G[32 st + 8 g4 .. + 7][16 T + c16], B = signs of
          // the same 8 bits of key 16 tau + c16 (none past 16 T)
          const bool on = 32 * st + 8 * g4 < 16 * T;
          uint4 ghi = make_uint4(0u, 0u, 0u, 0u), gmid = ghi, glo = ghi;
          if (on) {
            const float* gp = &sh.Gs[hm_gram_col<L>(16 * T + c16) + 32 * st + 8 * g4];
            split3(*reinterpret_cast<const float4*>(gp), *reinterpret_cast<const float4*>(gp + 4), ghi, gmid, glo);
          }
#pragma unroll
          for (int tau = 0; tau < 4; ++tau) {
            const uint32_t word = (uint32_t)__shfl((int)cws, 16 * tau + c16, 64);
            const uint4 sb = sign_operand((word >> (8 * g4)) & 0xFFu, on);
            ch[tau] = mfma32(ghi, sb, ch[tau]);
            as[tau] = mfma32(gmid, sb, as[tau]);
            as[tau] = mfma32(glo, sb, as[tau]);
          }
        }
      }
#pragma unroll
      for (int tau = 0; tau < 4; ++tau)
        *reinterpret_cast<float4*>(&Xs[(16 * tau + c16) * kHmXsStride + 4 * g4]) =
            make_float4((ah[tau][0] + as[tau][0]) + ch[tau][0], (ah[tau][1] + as[tau][1]) + ch[tau][1],
                        (ah[tau][2] + as[tau][2]) + ch[tau][2], (ah[tau][3] + as[tau][3]) + ch[tau][3]);
      wave_lds_sync();
      float y[16];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 v = *reinterpret_cast<const float4*>(&Xs[lane * kHmXsStride + 4 * q]);
        y[4 * q] = v.x, y[4 * q + 1] = v.y, y[4 * q + 2] = v.z, y[4 * q + 3] = v.w;
      }
      wave_lds_sync();
      // corrections by the bits of earlier blocks: y_j -= u_t Gr[t][j]
      // (on the vector units at L = 32)
#pragma unroll
      for (int w = 0; w < W; ++w) {
        if (hm_mm_corr<L>() || 32 * w >= 16 * T) break;
        const int nb = min(32, 16 * T - 32 * w);
        const uint32_t word = cw[w];
#pragma unroll 4
        for (int tt = 0; tt < nb; ++tt) {
          const float sg = ((word >> tt) & 1u) ? -1.f : 1.f;
          const int t = 32 * w + tt;
          const float4* gr = reinterpret_cast<const float4*>(&sh.Gs[hm_gram_at<L>(t, 16 * T)]);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float4 g = gr[q];
            y[4 * q] = fmaf(sg, g.x, y[4 * q]);
            y[4 * q + 1] = fmaf(sg, g.y, y[4 * q + 1]);
            y[4 * q + 2] = fmaf(sg, g.z, y[4 * q + 2]);
            y[4 * q + 3] = fmaf(sg, g.w, y[4 * q + 3]);
          }
        }
      }
      // The block's own bits, in order.  An uncertain decision takes the sign
      // of a^ for now and is recorded; the recorded ones are then decided in
      // the reference arithmetic, lowest bit first, and kept as overrides.
      // Where a speculated sign was wrong, the block's later bits of that key
      // rested on it, and the block is run again with the overrides.
      const float y0[16] = {y[0], y[1], y[2],  y[3],  y[4],  y[5],  y[6],  y[7],
                            y[8], y[9], y[10], y[11], y[12], y[13], y[14], y[15]};
      uint32_t ovm = 0u, ovv = 0u, ub = 0u;
      while (true) {
        uint32_t unc = 0u;
        ub = 0u;
#pragma unroll
        for (int i = 0; i < 16; ++i) y[i] = y0[i];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int bit = 16 * T + i;
          const float4 cb = sh.cst[bit];
          const float a = y[i];
          const float E = fmaf(nk * cb.x, cb.y, fmaf(cb.z, fabsf(a), cb.w + nkx)) * (1.f + 0x1p-8f);
          const bool sure = !valid || (fabsf(a) > E && E < 1e30f);
          bool u = a >= 0.f;
          if ((ovm >> i) & 1u) u = (ovv >> i) & 1u;
          else if (!sure) unc |= 1u << i;
          ub |= (u ? 1u : 0u) << i;
          if (i < 15) {
            const float sg = u ? -1.f : 1.f;
            const float4* gr = reinterpret_cast<const float4*>(&sh.Gs[hm_gram_diag<L>(bit)]);
#pragma unroll
            for (int q = (i + 1) / 4; q < 4; ++q) {
              const float4 g = gr[q];
              const float gv[4] = {g.x, g.y, g.z, g.w};
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if (4 * q + e > i) y[4 * q + e] = fmaf(sg, gv[e], y[4 * q + e]);
            }
          }
        }
        unsigned long long todo = __ballot(unc != 0u);
        if (!todo) break;
        bool rerun = false;
        while (todo) {
          const int j = __ffsll((long long)todo) - 1;
          todo &= todo - 1;
          uint32_t uj = __builtin_amdgcn_readlane(unc, j);
          const uint32_t ubj = __builtin_amdgcn_readlane(ub, j);
          uint32_t uw[4] = {0u, 0u, 0u, 0u};
#pragma unroll
          for (int w = 0; w < W; ++w) uw[w] = __builtin_amdgcn_readlane(cw[w], j);
          uw[(16 * T) >> 5] |= ubj << ((16 * T) & 31);
          // (the read-lane builtin returns a signed int: widen through uint32_t)
          const uint64_t rp = (uint64_t)(uintptr_t)my_row;
          const uint32_t rlo = (uint32_t)__builtin_amdgcn_readlane((uint32_t)rp, j);
          const uint32_t rhi = (uint32_t)__builtin_amdgcn_readlane((uint32_t)(rp >> 32), j);
          const uint16_t* krow = reinterpret_cast<const uint16_t*>((uintptr_t)(((uint64_t)rhi << 32) | rlo));
          while (uj) {
            const int i0 = __ffs(uj) - 1;
            uj &= uj - 1;
            const double ae = hm_reference_decision(krow, sh.Ps, 16 * T + i0, uw[0], uw[1], uw[2], uw[3], fb);
            const bool uref = ae >= 0.0;
            ++nfall;
            if (lane == j) {
              ovm |= 1u << i0;
              ovv |= (uref ? 1u : 0u) << i0;
              nfrag += fragile_decision(ae) ? 1u : 0u;
            }
            if (uref != (((ubj >> i0) & 1u) != 0u)) {
              rerun = true;  // this key's later bits of the block rested on the wrong sign
              break;
            }
          }
        }
        if (!rerun) break;
      }
      cw[(16 * T) >> 5] |= ub << ((16 * T) & 31);
    }
    if (valid) {
      uint32_t* cp = codes + b * sC_b + h * sC_h + (int64_t)(base + lane) * W;
      if constexpr (W == 1) cp[0] = cw[0];
      else if constexpr (W == 2) *reinterpret_cast<uint2*>(cp) = make_uint2(cw[0], cw[1]);
      else *reinterpret_cast<uint4*>(cp) = make_uint4(cw[0], cw[1], cw[2], cw[3]);
    }
  }
  // nfall is counted once per recomputed decision by every lane of the wavefront
  unsigned int wf = nfrag;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) wf += __shfl_xor(wf, o, 64);
  if (lane == 0) {
    if (wf) atomicAdd(&sh.nfrag, wf);
    if (nfall) atomicAdd(&sh.nfall, nfall);
  }
  __syncthreads();
  if (tid == 0) {
    if (fragile && sh.nfrag) atomicAdd(fragile, (unsigned long long)sh.nfrag);
    if (fallbacks && sh.nfall) atomicAdd(fallbacks, (unsigned long long)sh.nfall);
  }
}

template <int L>
static hipError_t launch_hash_mm_L(const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n, int B, int Hkv,
                                   int N, const float* P, int64_t sP_b, int64_t sP_h, uint32_t* codes, int64_t sC_b,
                                   int64_t sC_h, unsigned long long* fragile, unsigned long long* fallbacks,
                                   hipStream_t stream) {
  static_assert(sizeof(HmShared<L>) <= 160 * 1024, "LDS budget");
  constexpr int kHmThreads = hm_threads<L>();
  // about 2048 workgroups in all, each over whole wavefront iterations
  const long long total = (long long)B * Hkv * N;
  long long per = (total + 2047) / 2048;
  per = (per + kHmThreads - 1) / kHmThreads * kHmThreads;
  per = per < kHmThreads ? kHmThreads : per > 64 * kHmThreads ? 64 * kHmThreads : per;
  const int keys_per_wg = (int)per;
  const dim3 grid((unsigned)((N + keys_per_wg - 1) / keys_per_wg), (unsigned)(B * Hkv));
  hash_mm_kernel<L><<<grid, kHmThreads, 0, stream>>>(K, sK_b, sK_h, sK_n, Hkv, N, P, sP_b, sP_h, codes, sC_b,
                                                        sC_h, fragile, fallbacks, keys_per_wg);
  return hipGetLastError();
}

hipError_t launch_hash_mm(const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n, int B, int Hkv, int N, int L,
                          const float* P, int64_t sP_b, int64_t sP_h, uint32_t* codes, int64_t sC_b, int64_t sC_h,
                          unsigned long long* fragile, unsigned long long* fallbacks, hipStream_t stream) {
  switch (L) {
    case 32:
      return launch_hash_mm_L<32>(K, sK_b, sK_h, sK_n, B, Hkv, N, P, sP_b, sP_h, codes, sC_b, sC_h, fragile,
                                  fallbacks, stream);
    case 64:
      return launch_hash_mm_L<64>(K, sK_b, sK_h, sK_n, B, Hkv, N, P, sP_b, sP_h, codes, sC_b, sC_h, fragile,
                                  fallbacks, stream);
    default:
      return launch_hash_mm_L<128>(K, sK_b, sK_h, sK_n, B, Hkv, N, P, sP_b, sP_h, codes, sC_b, sC_h, fragile,
                                   fallbacks, stream);
  }
}

}  // namespace bpc
