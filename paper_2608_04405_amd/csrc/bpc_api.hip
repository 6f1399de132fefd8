// Host side of the C ABI: argument checks, workspace layouts, dispatch.
//
// Every check runs before anything is enqueued, so a call that returns an
// error has launched nothing and written no output.

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "bpc_internal.h"

namespace bpc {

static thread_local char g_last_error[512] = "";

static int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return status;
}

static int hip_fail(hipError_t e, const char* what) {
  return fail(BPC_EHIP, "%s: %s", what, hipGetErrorString(e));
}

static size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
static bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

static int check_code_len(int L) {
  if (L != 32 && L != 64 && L != 128) return fail(BPC_EUNSUPPORTED, "L=%d: code length must be 32, 64 or 128", L);
  return BPC_OK;
}

static int check_head_dim(int D) {
  if (D != kHeadDim) return fail(BPC_EUNSUPPORTED, "D=%d: only head_dim 128 is supported", D);
  return BPC_OK;
}

// A bf16 [B, H, >=N, D] tensor given by strides.
static int check_kv(const char* name, const uint16_t* p, int64_t sb, int64_t sh, int64_t sn) {
  if (!p) return fail(BPC_EINVAL, "%s is NULL", name);
  if (sb < 0 || sh < 0 || sn < kHeadDim)
    return fail(BPC_EINVAL, "%s strides (%lld, %lld, %lld) invalid: need s_b, s_h >= 0 and s_n >= 128", name,
                (long long)sb, (long long)sh, (long long)sn);
  if (!aligned16(p) || (sb % 8) || (sh % 8) || (sn % 8))
    return fail(BPC_EALIGN, "%s must be 16-byte aligned with strides multiple of 8 elements", name);
  return BPC_OK;
}

static int check_codes(const char* name, const void* p, int64_t sb, int64_t sh, int W) {
  if (!p) return fail(BPC_EINVAL, "%s is NULL", name);
  if (sb < 0 || sh < 0) return fail(BPC_EINVAL, "%s strides must be >= 0", name);
  if (!aligned16(p) || (sb % W) || (sh % W))
    return fail(BPC_EALIGN, "%s must be 16-byte aligned with strides multiple of W=%d words", name, W);
  return BPC_OK;
}

static int check_proj(const float* P, int64_t sb, int64_t sh) {
  if (!P) return fail(BPC_EINVAL, "P is NULL");
  if (sb < 0 || sh < 0) return fail(BPC_EINVAL, "P strides must be >= 0");
  if (!aligned16(P) || (sb % 4) || (sh % 4))
    return fail(BPC_EALIGN, "P must be 16-byte aligned with strides multiple of 4 floats");
  return BPC_OK;
}

static int check_opt_aligned(const char* name, const void* p) {
  if (p && !aligned16(p)) return fail(BPC_EALIGN, "%s must be 16-byte aligned", name);
  return BPC_OK;
}

DecodeLayout decode_layout(int B, int Hq, int Hkv, int N, int L, int k) {
  DecodeLayout d{};
  const size_t BH = (size_t)B * Hkv;
  d.W = L / 32;
  d.G = Hq / Hkv;
  const int fused_slice = decode_fused_slice(B, Hq, Hkv, N, L);
  d.fused = fused_slice != 0;
  d.slice = d.fused ? fused_slice : kSlice;
  d.nslices = (N + d.slice - 1) / d.slice;
  const size_t S = BH * d.nslices;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align_up(o + bytes, 256);
    return at;
  };
  d.off_sync = take(kSyncRegionBytes);  // both paths; only the fused one uses it
  if (d.fused) {
    d.off_pub = take(S * kFusedPubWords * sizeof(uint32_t));
    d.off_part = take(S * d.G * (kHeadDim + 2) * sizeof(float));
    d.off_rows = take(BH * (size_t)k * sizeof(int32_t));
    d.total = o;
    return d;
  }
  d.off_cand = take(S * (size_t)kSlice * sizeof(uint32_t));
  d.off_meta = take(S * 4 * sizeof(uint32_t));
  d.off_hist_fine = take(S * (size_t)fine_stride(L) * sizeof(uint32_t));
  d.off_hist_cc = take(S * (size_t)kCoarseStride * sizeof(uint32_t));
  d.off_win = take(S * (size_t)kWinRec * sizeof(uint32_t));
  d.off_part = take(S * d.G * (kHeadDim + 2) * sizeof(float));
  d.off_qcode = take(BH * kQcodeStride * sizeof(uint32_t));
  d.total = o;
  return d;
}

BuildLayout build_layout(int B, int Hkv, int N, int L) {
  BuildLayout b{};
  const size_t BH = (size_t)B * Hkv;
  b.nchunks = (N + kBuildChunk - 1) / kBuildChunk;
  size_t o = 0;
  b.off_part = o;  // one fp64 tree sum per chunk and coordinate
  o = align_up(o + BH * b.nchunks * (size_t)kHeadDim * sizeof(double), 256);
  b.nfold = b.nchunks > 8 * kBuildFold ? (b.nchunks + kBuildFold - 1) / kBuildFold : 0;
  b.off_fold = o;  // one fp64 tree sum per block of chunks and coordinate
  o = align_up(o + BH * b.nfold * (size_t)kHeadDim * sizeof(double), 256);
  b.off_p64 = o;   // P widened to fp64, the scalar operand of the residual
  o = align_up(o + BH * (size_t)L * kHeadDim * sizeof(double), 256);
  b.off_g64 = o;   // G widened to fp64
  o = align_up(o + (size_t)L * kHeadDim * sizeof(double), 256);
  b.total = o;
  b.off_ck = o;    // fp64 residual of every key, padded to whole chunks
  o = align_up(o + BH * b.nchunks * (size_t)kBuildChunk * kHeadDim * sizeof(double), 256);
  b.total_ck = o;
  return b;
}

static int check_sizes(int B, int Hkv, int N) {
  if (B < 1 || Hkv < 1 || N < 1) return fail(BPC_EINVAL, "B=%d, Hkv=%d, N=%d must all be >= 1", B, Hkv, N);
  if ((int64_t)N > (int64_t)(1 << 30)) return fail(BPC_EINVAL, "N=%d too large", N);
  return BPC_OK;
}

}  // namespace bpc

using namespace bpc;

extern "C" {

const char* bpc_status_string(int status) {
  switch (status) {
    case BPC_OK: return "ok";
    case BPC_EINVAL: return "invalid argument";
    case BPC_EUNSUPPORTED: return "unsupported shape";
    case BPC_EALIGN: return "misaligned pointer or stride";
    case BPC_EWORKSPACE: return "workspace missing or too small";
    case BPC_EHIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* bpc_last_error(void) { return g_last_error; }

int bpc_version(void) { return 200; }

int bpc_set_decode_path(int path) {
  if (path < 0 || path > 2)
    return fail(BPC_EINVAL, "path=%d must be 0 (automatic), 1 (three launches) or 2 (fused, large slices only)", path);
  decode_set_path(path);
  return BPC_OK;
}

int bpc_decode_slice_keys(int B, int Hq, int Hkv, int N, int L) {
  if (B < 1 || Hq < 1 || Hkv < 1 || N < 1 || (L != 32 && L != 64 && L != 128)) return 0;
  const int sl = decode_fused_slice(B, Hq, Hkv, N, L);
  return sl ? sl : kSlice;
}

int bpc_decode_path_taken(int B, int Hq, int Hkv, int N, int L) {
  if (B < 1 || Hq < 1 || Hkv < 1 || N < 1 || (L != 32 && L != 64 && L != 128)) return 1;
  return decode_fused_ok(B, Hq, Hkv, N, L) ? 0 : 1;
}

size_t bpc_build_workspace_bytes(int B, int Hkv, int N, int D, int L) {
  if (B < 1 || Hkv < 1 || N < 1 || D != kHeadDim) return 0;
  return build_layout(B, Hkv, N, L).total;
}

size_t bpc_build_checkpoint_workspace_bytes(int B, int Hkv, int N, int D, int L) {
  if (B < 1 || Hkv < 1 || N < 1 || D != kHeadDim) return 0;
  return build_layout(B, Hkv, N, L).total_ck;
}

int bpc_build_hash(const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n, int B, int Hkv, int N,
                   int D, int L, const float* G, float* P_out, uint32_t* codes_out, int64_t sC_b,
                   int64_t sC_h, float* err_out, unsigned long long* fragile_out, void* workspace,
                   size_t workspace_bytes, void* stream) {
  g_last_error[0] = 0;
  int st;
  if ((st = check_sizes(B, Hkv, N))) return st;
  if ((st = check_head_dim(D))) return st;
  if ((st = check_code_len(L))) return st;
  if ((st = check_kv("K", K, sK_b, sK_h, sK_n))) return st;
  if (!G || !P_out) return fail(BPC_EINVAL, "G and P_out are required");
  if (!aligned16(G) || !aligned16(P_out)) return fail(BPC_EALIGN, "G and P_out must be 16-byte aligned");
  if ((st = check_codes("codes_out", codes_out, sC_b, sC_h, L / 32))) return st;
  if ((st = check_opt_aligned("err_out", err_out))) return st;
  const BuildLayout lay = build_layout(B, Hkv, N, L);
  if (!workspace || workspace_bytes < lay.total)
    return fail(BPC_EWORKSPACE, "workspace of %zu bytes given, %zu needed", workspace ? workspace_bytes : 0,
                lay.total);
  if (reinterpret_cast<uintptr_t>(workspace) & 255u) return fail(BPC_EALIGN, "workspace must be 256-byte aligned");
  const bool checkpoint = workspace_bytes >= lay.total_ck;
  hipError_t e = launch_build(K, sK_b, sK_h, sK_n, B, Hkv, N, L, G, P_out, codes_out, sC_b, sC_h, err_out,
                              fragile_out, static_cast<char*>(workspace), checkpoint,
                              static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "bpc_build_hash launch");
  return BPC_OK;
}

int bpc_hash_keys(const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n, int B, int Hkv, int N, int D,
                  int L, const float* P, int64_t sP_b, int64_t sP_h, uint32_t* codes_out, int64_t sC_b,
                  int64_t sC_h, float* err_out, unsigned long long* fragile_out, void* stream) {
  g_last_error[0] = 0;
  int st;
  if ((st = check_sizes(B, Hkv, N))) return st;
  if ((st = check_head_dim(D))) return st;
  if ((st = check_code_len(L))) return st;
  if ((st = check_kv("K", K, sK_b, sK_h, sK_n))) return st;
  if ((st = check_proj(P, sP_b, sP_h))) return st;
  if ((st = check_codes("codes_out", codes_out, sC_b, sC_h, L / 32))) return st;
  if ((st = check_opt_aligned("err_out", err_out))) return st;
  hipError_t e = launch_hash(K, sK_b, sK_h, sK_n, B, Hkv, N, L, P, sP_b, sP_h, codes_out, sC_b, sC_h, err_out,
                             fragile_out, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "bpc_hash_keys launch");
  return BPC_OK;
}

int bpc_hash_keys_mm(const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n, int B, int Hkv, int N, int D,
                     int L, const float* P, int64_t sP_b, int64_t sP_h, uint32_t* codes_out, int64_t sC_b,
                     int64_t sC_h, unsigned long long* fragile_out, unsigned long long* fallbacks_out, void* stream) {
  g_last_error[0] = 0;
  int st;
  if ((st = check_sizes(B, Hkv, N))) return st;
  if ((st = check_head_dim(D))) return st;
  if ((st = check_code_len(L))) return st;
  if ((st = check_kv("K", K, sK_b, sK_h, sK_n))) return st;
  if ((st = check_proj(P, sP_b, sP_h))) return st;
  if ((st = check_codes("codes_out", codes_out, sC_b, sC_h, L / 32))) return st;
  hipError_t e = launch_hash_mm(K, sK_b, sK_h, sK_n, B, Hkv, N, L, P, sP_b, sP_h, codes_out, sC_b, sC_h, fragile_out,
                                fallbacks_out, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "bpc_hash_keys_mm launch");
  return BPC_OK;
}

int bpc_append_kv(const uint16_t* k_new, int64_t sKn_b, int64_t sKn_h, int64_t sKn_t, const uint16_t* v_new,
                  int64_t sVn_b, int64_t sVn_h, int64_t sVn_t, uint16_t* K, int64_t sK_b, int64_t sK_h,
                  int64_t sK_n, uint16_t* V, int64_t sV_b, int64_t sV_h, int64_t sV_n, uint32_t* codes,
                  int64_t sC_b, int64_t sC_h, const float* P, int64_t sP_b, int64_t sP_h, int B, int Hkv,
                  int Ncap, int pos, int T, int D, int L, float* err_out, unsigned long long* fragile_out,
                  void* stream) {
  g_last_error[0] = 0;
  int st;
  if ((st = check_sizes(B, Hkv, Ncap))) return st;
  if (T < 1 || pos < 0 || (int64_t)pos + T > Ncap)
    return fail(BPC_EINVAL, "pos=%d, T=%d must satisfy pos >= 0, T >= 1, pos + T <= Ncap=%d", pos, T, Ncap);
  if ((st = check_head_dim(D))) return st;
  if ((st = check_code_len(L))) return st;
  if ((st = check_kv("k_new", k_new, sKn_b, sKn_h, sKn_t))) return st;
  if ((st = check_kv("v_new", v_new, sVn_b, sVn_h, sVn_t))) return st;
  if ((st = check_kv("K", K, sK_b, sK_h, sK_n))) return st;
  if ((st = check_kv("V", V, sV_b, sV_h, sV_n))) return st;
  if ((st = check_proj(P, sP_b, sP_h))) return st;
  if ((st = check_codes("codes", codes, sC_b, sC_h, L / 32))) return st;
  if ((st = check_opt_aligned("err_out", err_out))) return st;
  AppendCopy cp{};
  cp.Kc = K + (int64_t)pos * sK_n, cp.sKc_b = sK_b, cp.sKc_h = sK_h, cp.sKc_n = sK_n;
  cp.Vn = v_new, cp.sVn_b = sVn_b, cp.sVn_h = sVn_h, cp.sVn_n = sVn_t;
  cp.Vc = V + (int64_t)pos * sV_n, cp.sVc_b = sV_b, cp.sVc_h = sV_h, cp.sVc_n = sV_n;
  hipError_t e = launch_hash(k_new, sKn_b, sKn_h, sKn_t, B, Hkv, T, L, P, sP_b, sP_h, codes + (int64_t)pos * (L / 32),
                             sC_b, sC_h, err_out, fragile_out, static_cast<hipStream_t>(stream), &cp);
  if (e != hipSuccess) return hip_fail(e, "bpc_append_kv launch");
  return BPC_OK;
}

size_t bpc_decode_workspace_bytes(int B, int Hq, int Hkv, int N, int D, int L, int k) {
  if (B < 1 || Hkv < 1 || Hq < Hkv || Hq % Hkv || N < 1 || k < 1 || k > N || D != kHeadDim) return 0;
  if (L != 32 && L != 64 && L != 128) return 0;
  return decode_layout(B, Hq, Hkv, N, L, k).total;
}

static int decode_impl(const uint16_t* q, const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                       const uint16_t* V, int64_t sV_b, int64_t sV_h, int64_t sV_n, const uint32_t* codes,
                       int64_t sC_b, int64_t sC_h, const float* P, int64_t sP_b, int64_t sP_h, int B, int Hq,
                       int Hkv, int N, int D, int L, int k, float sm_scale, float* out, int32_t* idx_out,
                       int32_t* score_out, uint32_t* qcode_out, const int32_t* serr, int64_t sS_b, int64_t sS_h,
                       int m, int32_t* added_out, void* workspace, size_t workspace_bytes, void* stream,
                       void* const* events, int n_events, bool launch = true) {
  g_last_error[0] = 0;
  int st;
  if ((st = check_sizes(B, Hkv, N))) return st;
  if (Hq < Hkv || Hq % Hkv) return fail(BPC_EINVAL, "Hq=%d must be a positive multiple of Hkv=%d", Hq, Hkv);
  {
    const int G = Hq / Hkv;
    if (G > kMaxGroup || (G & (G - 1)))
      return fail(BPC_EUNSUPPORTED, "group size Hq/Hkv=%d must be 1, 2, 4, 8 or 16", G);
  }
  if ((st = check_head_dim(D))) return st;
  if ((st = check_code_len(L))) return st;
  if (k < 1 || k > N) return fail(BPC_EINVAL, "k=%d must satisfy 1 <= k <= N=%d", k, N);
  if ((int64_t)N > (int64_t)kMaxSlices * kSlice)
    return fail(BPC_EUNSUPPORTED, "N=%d: decode supports at most %d cached keys per head", N, kMaxSlices * kSlice);
  if (!(sm_scale > 0.0f) || !__builtin_isfinite(sm_scale))
    return fail(BPC_EINVAL, "sm_scale must be finite and > 0");
  if (!q || !out) return fail(BPC_EINVAL, "q and out are required");
  if (!aligned16(q) || !aligned16(out)) return fail(BPC_EALIGN, "q and out must be 16-byte aligned");
  if ((st = check_kv("K", K, sK_b, sK_h, sK_n))) return st;
  if ((st = check_kv("V", V, sV_b, sV_h, sV_n))) return st;
  // the attention kernel addresses a row by a 32-bit byte offset within its head
  if ((int64_t)(N - 1) * sK_n * 2 + 256 > (int64_t)UINT32_MAX || (int64_t)(N - 1) * sV_n * 2 + 256 > (int64_t)UINT32_MAX)
    return fail(BPC_EUNSUPPORTED, "the N rows of one head must span less than 4 GiB (N=%d, row strides %lld, %lld)",
                N, (long long)sK_n, (long long)sV_n);
  if ((st = check_codes("codes", codes, sC_b, sC_h, L / 32))) return st;
  if ((st = check_proj(P, sP_b, sP_h))) return st;
  if ((st = check_opt_aligned("idx_out", idx_out))) return st;
  if ((st = check_opt_aligned("score_out", score_out))) return st;
  if ((st = check_opt_aligned("qcode_out", qcode_out))) return st;
  if (m < 0 || m > N) return fail(BPC_EINVAL, "m=%d must satisfy 0 <= m <= N=%d", m, N);
  if (m > 0) {
    if (!serr) return fail(BPC_EINVAL, "serr is required when m > 0");
    if (sS_b < 0 || sS_h < 0) return fail(BPC_EINVAL, "serr strides must be >= 0");
    if (!aligned4(serr)) return fail(BPC_EALIGN, "serr must be 4-byte aligned");
    if ((st = check_opt_aligned("added_out", added_out))) return st;
  }
  if (events && n_events != BPC_DECODE_STAGES + 1)
    return fail(BPC_EINVAL, "n_events=%d, expected %d", n_events, BPC_DECODE_STAGES + 1);
  const DecodeLayout lay = decode_layout(B, Hq, Hkv, N, L, k);
  if (!workspace || workspace_bytes < lay.total)
    return fail(BPC_EWORKSPACE, "workspace of %zu bytes given, %zu needed", workspace ? workspace_bytes : 0,
                lay.total);
  if (reinterpret_cast<uintptr_t>(workspace) & 255u) return fail(BPC_EALIGN, "workspace must be 256-byte aligned");
  if (!launch) return BPC_OK;

  DecodeArgs a{};
  a.q = q;
  a.K = K, a.sK_b = sK_b, a.sK_h = sK_h, a.sK_n = sK_n;
  a.V = V, a.sV_b = sV_b, a.sV_h = sV_h, a.sV_n = sV_n;
  a.codes = codes, a.sC_b = sC_b, a.sC_h = sC_h;
  a.P = P, a.sP_b = sP_b, a.sP_h = sP_h;
  a.B = B, a.Hq = Hq, a.Hkv = Hkv, a.N = N, a.L = L, a.k = k;
  a.sm_scale = sm_scale;
  a.out = out, a.idx_out = idx_out, a.score_out = score_out, a.qcode_out = qcode_out;
  a.serr = m > 0 ? serr : nullptr, a.sS_b = sS_b, a.sS_h = sS_h, a.m = m, a.added_out = m > 0 ? added_out : nullptr;
  a.ws = static_cast<char*>(workspace);
  a.stream = static_cast<hipStream_t>(stream);
  a.events = reinterpret_cast<hipEvent_t const*>(events);
  hipError_t e = launch_decode(a, lay);
  if (e != hipSuccess) return hip_fail(e, "bpc_decode_attention launch");
  return BPC_OK;
}

int bpc_decode_attention(const uint16_t* q, const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                         const uint16_t* V, int64_t sV_b, int64_t sV_h, int64_t sV_n, const uint32_t* codes,
                         int64_t sC_b, int64_t sC_h, const float* P, int64_t sP_b, int64_t sP_h, int B, int Hq,
                         int Hkv, int N, int D, int L, int k, float sm_scale, float* out, int32_t* idx_out,
                         int32_t* score_out, uint32_t* qcode_out, void* workspace, size_t workspace_bytes,
                         void* stream) {
  return decode_impl(q, K, sK_b, sK_h, sK_n, V, sV_b, sV_h, sV_n, codes, sC_b, sC_h, P, sP_b, sP_h, B, Hq, Hkv,
                     N, D, L, k, sm_scale, out, idx_out, score_out, qcode_out, nullptr, 0, 0, 0, nullptr, workspace,
                     workspace_bytes, stream, nullptr, 0);
}

int bpc_decode_attention_eas(const uint16_t* q, const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                             const uint16_t* V, int64_t sV_b, int64_t sV_h, int64_t sV_n, const uint32_t* codes,
                             int64_t sC_b, int64_t sC_h, const float* P, int64_t sP_b, int64_t sP_h, int B, int Hq,
                             int Hkv, int N, int D, int L, int k, float sm_scale, const int32_t* serr, int64_t sS_b,
                             int64_t sS_h, int m, float* out, int32_t* idx_out, int32_t* added_out,
                             void* workspace, size_t workspace_bytes, void* stream) {
  return decode_impl(q, K, sK_b, sK_h, sK_n, V, sV_b, sV_h, sV_n, codes, sC_b, sC_h, P, sP_b, sP_h, B, Hq, Hkv,
                     N, D, L, k, sm_scale, out, idx_out, nullptr, nullptr, serr, sS_b, sS_h, m, added_out, workspace,
                     workspace_bytes, stream, nullptr, 0);
}

size_t bpc_decode_per_head_workspace_bytes(int B, int Hq, int Hkv, int N, int D, int L, int k) {
  if (B < 1 || Hkv < 1 || Hq < Hkv || Hq % Hkv || N < 1 || k < 1 || k > N || D != kHeadDim) return 0;
  if (L != 32 && L != 64 && L != 128) return 0;
  const int G = Hq / Hkv;
  return decode_layout(B * Hkv, G, G, N, L, k).total;
}

// Per-query-head selection runs the decode path with one query per "KV
// head": the G query heads of (b, h) become G heads of a sequence b' that
// all read (b, h)'s K, V, codes and P (head stride 0).  When every tensor's
// batch stride is Hkv times its head stride, b' = b Hkv + h addresses all
// of them linearly and one call covers the batch; otherwise each sequence
// is one call.
int bpc_decode_attention_per_head(const uint16_t* q, const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                                  const uint16_t* V, int64_t sV_b, int64_t sV_h, int64_t sV_n,
                                  const uint32_t* codes, int64_t sC_b, int64_t sC_h, const float* P, int64_t sP_b,
                                  int64_t sP_h, int B, int Hq, int Hkv, int N, int D, int L, int k, float sm_scale,
                                  float* out, int32_t* idx_out, int32_t* score_out, uint32_t* qcode_out,
                                  void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error[0] = 0;
  int st;
  if ((st = check_sizes(B, Hkv, N))) return st;
  if (Hq < Hkv || Hq % Hkv) return fail(BPC_EINVAL, "Hq=%d must be a positive multiple of Hkv=%d", Hq, Hkv);
  if ((int64_t)B * Hkv > (int64_t)(1 << 20)) return fail(BPC_EINVAL, "B*Hkv=%lld too large", (long long)B * Hkv);
  if ((st = check_kv("K", K, sK_b, sK_h, sK_n))) return st;
  if ((st = check_kv("V", V, sV_b, sV_h, sV_n))) return st;
  if ((st = check_code_len(L))) return st;
  if ((st = check_codes("codes", codes, sC_b, sC_h, L / 32))) return st;
  if ((st = check_proj(P, sP_b, sP_h))) return st;
  const size_t need = bpc_decode_per_head_workspace_bytes(B, Hq, Hkv, N, D, L, k);
  if (need && (!workspace || workspace_bytes < need))
    return fail(BPC_EWORKSPACE, "workspace of %zu bytes given, %zu needed", workspace ? workspace_bytes : 0, need);
  const int G = Hq / Hkv;
  const bool linear = sK_b == Hkv * sK_h && sV_b == Hkv * sV_h && sC_b == Hkv * sC_h && sP_b == Hkv * sP_h;
  const int calls = linear ? 1 : B;
  const int Bc = linear ? B * Hkv : Hkv;  // sequences b' per call
  const int W = L / 32;
  // every call's offset pointers are checked (alignment included) before
  // the first one launches, so that an error leaves every output untouched
  for (int pass = 0; pass < 2; ++pass)
    for (int c = 0; c < calls; ++c) {
      st = decode_impl(q + (size_t)c * Hq * kHeadDim, K + c * sK_b, sK_h, 0, sK_n, V + c * sV_b, sV_h, 0, sV_n,
                       codes + c * sC_b, sC_h, 0, P + c * sP_b, sP_h, 0, Bc, G, G, N, D, L, k, sm_scale,
                       out + (size_t)c * Hq * kHeadDim, idx_out ? idx_out + (size_t)c * Hq * k : nullptr,
                       score_out ? score_out + (size_t)c * Hq * N : nullptr,
                       qcode_out ? qcode_out + (size_t)c * Hq * 8 * W : nullptr, nullptr, 0, 0, 0, nullptr,
                       workspace, workspace_bytes, stream, nullptr, 0, pass == 1);
      if (st) {
        if (calls > 1) {
          char detail[sizeof(g_last_error)];
          snprintf(detail, sizeof(detail), "%s", g_last_error);
          return fail(st, "sequence %d of %d (one call per sequence): %s", c, calls, detail);
        }
        return st;
      }
    }
  return BPC_OK;
}

size_t bpc_dense_workspace_bytes(int B, int Hq, int Hkv, int N, int D) {
  if (B < 1 || Hkv < 1 || Hq < Hkv || Hq % Hkv || N < 1 || D != kHeadDim) return 0;
  const size_t nchunks = ((size_t)N + kSlice - 1) / kSlice;
  return align_up((size_t)B * Hkv * nchunks * (Hq / Hkv) * (kHeadDim + 2) * sizeof(float), 256);
}

int bpc_dense_attention(const uint16_t* q, const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                        const uint16_t* V, int64_t sV_b, int64_t sV_h, int64_t sV_n, int B, int Hq, int Hkv, int N,
                        int D, float sm_scale, float* out, void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error[0] = 0;
  int st;
  if ((st = check_sizes(B, Hkv, N))) return st;
  if (Hq < Hkv || Hq % Hkv) return fail(BPC_EINVAL, "Hq=%d must be a positive multiple of Hkv=%d", Hq, Hkv);
  {
    const int G = Hq / Hkv;
    if (G > kMaxGroup || (G & (G - 1)))
      return fail(BPC_EUNSUPPORTED, "group size Hq/Hkv=%d must be 1, 2, 4, 8 or 16", G);
  }
  if ((st = check_head_dim(D))) return st;
  if ((int64_t)N > (int64_t)kMaxSlices * kSlice)
    return fail(BPC_EUNSUPPORTED, "N=%d: at most %d cached keys per head", N, kMaxSlices * kSlice);
  if (!(sm_scale > 0.0f) || !__builtin_isfinite(sm_scale))
    return fail(BPC_EINVAL, "sm_scale must be finite and > 0");
  if (!q || !out) return fail(BPC_EINVAL, "q and out are required");
  if (!aligned16(q) || !aligned16(out)) return fail(BPC_EALIGN, "q and out must be 16-byte aligned");
  if ((st = check_kv("K", K, sK_b, sK_h, sK_n))) return st;
  if ((st = check_kv("V", V, sV_b, sV_h, sV_n))) return st;
  if ((int64_t)(N - 1) * sK_n * 2 + 256 > (int64_t)UINT32_MAX || (int64_t)(N - 1) * sV_n * 2 + 256 > (int64_t)UINT32_MAX)
    return fail(BPC_EUNSUPPORTED, "the N rows of one head must span less than 4 GiB");
  const size_t need = bpc_dense_workspace_bytes(B, Hq, Hkv, N, D);
  if (!workspace || workspace_bytes < need)
    return fail(BPC_EWORKSPACE, "workspace of %zu bytes given, %zu needed", workspace ? workspace_bytes : 0, need);
  if (reinterpret_cast<uintptr_t>(workspace) & 255u) return fail(BPC_EALIGN, "workspace must be 256-byte aligned");
  DenseArgs a{};
  a.q = q;
  a.K = K, a.sK_b = sK_b, a.sK_h = sK_h, a.sK_n = sK_n;
  a.V = V, a.sV_b = sV_b, a.sV_h = sV_h, a.sV_n = sV_n;
  a.B = B, a.Hq = Hq, a.Hkv = Hkv, a.N = N, a.sm_scale = sm_scale, a.out = out;
  a.ws = static_cast<char*>(workspace);
  a.stream = static_cast<hipStream_t>(stream);
  hipError_t e = launch_dense(a);
  if (e != hipSuccess) return hip_fail(e, "bpc_dense_attention launch");
  return BPC_OK;
}

int bpc_select_hard(const float* err, int64_t sE_b, int64_t sE_h, int B, int Hkv, int N, int m, int32_t* serr_out,
                    void* stream) {
  g_last_error[0] = 0;
  int st;
  if ((st = check_sizes(B, Hkv, N))) return st;
  if (m < 0 || m > N) return fail(BPC_EINVAL, "m=%d must satisfy 0 <= m <= N=%d", m, N);
  if (m == 0) return BPC_OK;
  if (!err || !serr_out) return fail(BPC_EINVAL, "err and serr_out are required");
  if (sE_b < 0 || sE_h < 0) return fail(BPC_EINVAL, "err strides must be >= 0");
  if (!aligned4(err) || !aligned4(serr_out)) return fail(BPC_EALIGN, "err and serr_out must be 4-byte aligned");
  hipError_t e = launch_select_hard(err, sE_b, sE_h, B, Hkv, N, m, serr_out, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "bpc_select_hard launch");
  return BPC_OK;
}

// ---------------------------------------------------------------------------
// Decode without a caller workspace: the workspace is `scratch`, a static
// device array of kScratchBytes that every GPU the library runs on holds
// until the process ends.  In host code `scratch` only names the symbol; its
// device address on the current GPU comes from hipGetSymbolAddress, once per
// device, and only that address is ever passed to kernels.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = size_t(64) << 20;
constexpr int kScratchDevices = 64;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kScratchDevices];

// The scratch address on the GPU of `stream` (which must be the current
// device); looked up on the first call on that device.
static int scratch_for(void* stream, void** ptr) {
  int dev = -1, sdev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  e = hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev);
  if (e != hipSuccess) return hip_fail(e, "hipStreamGetDevice");
  if (sdev != dev) return fail(BPC_EINVAL, "the stream belongs to device %d, the current device is %d", sdev, dev);
  if (dev < 0 || dev >= kScratchDevices) return fail(BPC_EUNSUPPORTED, "device %d: at most %d devices", dev, kScratchDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(BPC_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return BPC_OK;
}

size_t bpc_decode_noalloc_max_bytes(void) { return kScratchBytes; }

int bpc_decode_attention_noalloc(const uint16_t* q, const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                                 const uint16_t* V, int64_t sV_b, int64_t sV_h, int64_t sV_n,
                                 const uint32_t* codes, int64_t sC_b, int64_t sC_h, const float* P, int64_t sP_b,
                                 int64_t sP_h, int B, int Hq, int Hkv, int N, int D, int L, int k, float sm_scale,
                                 float* out, int32_t* idx_out, int32_t* score_out, uint32_t* qcode_out,
                                 void* stream) {
  g_last_error[0] = 0;
  const size_t need = bpc_decode_workspace_bytes(B, Hq, Hkv, N, D, L, k);
  if (need > kScratchBytes)
    return fail(BPC_EWORKSPACE, "this decode needs %zu bytes of scratch; the static scratch holds %zu (%zu MiB)",
                need, kScratchBytes, kScratchBytes >> 20);
  void* ws = nullptr;
  int st = scratch_for(stream, &ws);
  if (st) return st;
  return decode_impl(q, K, sK_b, sK_h, sK_n, V, sV_b, sV_h, sV_n, codes, sC_b, sC_h, P, sP_b, sP_h, B, Hq, Hkv,
                     N, D, L, k, sm_scale, out, idx_out, score_out, qcode_out, nullptr, 0, 0, 0, nullptr, ws,
                     kScratchBytes, stream, nullptr, 0);
}

int bpc_decode_attention_profiled(const uint16_t* q, const uint16_t* K, int64_t sK_b, int64_t sK_h,
                                  int64_t sK_n, const uint16_t* V, int64_t sV_b, int64_t sV_h, int64_t sV_n,
                                  const uint32_t* codes, int64_t sC_b, int64_t sC_h, const float* P,
                                  int64_t sP_b, int64_t sP_h, int B, int Hq, int Hkv, int N, int D, int L, int k,
                                  float sm_scale, float* out, int32_t* idx_out, int32_t* score_out,
                                  uint32_t* qcode_out, void* workspace, size_t workspace_bytes, void* stream,
                                  void* const* events, int n_events) {
  if (!events) return fail(BPC_EINVAL, "events is NULL");
  for (int i = 0; i < n_events; ++i)
    if (!events[i]) return fail(BPC_EINVAL, "events[%d] is NULL", i);
  return decode_impl(q, K, sK_b, sK_h, sK_n, V, sV_b, sV_h, sV_n, codes, sC_b, sC_h, P, sP_b, sP_h, B, Hq, Hkv,
                     N, D, L, k, sm_scale, out, idx_out, score_out, qcode_out, nullptr, 0, 0, 0, nullptr, workspace,
                     workspace_bytes, stream, events, n_events);
}

}  // extern "C"
