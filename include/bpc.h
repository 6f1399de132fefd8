/*
 * bpc.h -- C ABI of the BinaryPC decode hot path on AMD Instinct MI355X
 * (gfx950).
 *
 * BinaryPC ("Training-Free Hashing-Based Attention via Binary Principal
 * Components") approximates every cached key k by h P, with a binary code
 * h in {-1,+1}^L and a real projection P [L, D] (Sec. 3.2, Problem
 * Formulation).  At prefill, P and the codes are built greedily from the
 * keys (Algorithm "Constructing hash codes and corresponding hashing
 * projection"), or keys are hashed against a given P (Algorithm "Given
 * projection, computing hashcode").  At decode, the query is projected to
 * q P^T, quantised to 7-bit magnitudes and packed into bit planes; every
 * cached code is scored with XOR and popcount (Algorithm "Computing hashing
 * score", Appendix "CUDA Optimizations on Bitwise Operations"); the top-k
 * keys are selected and softmax attention runs over the gathered K/V rows
 * only (Sec. 4.2, Kernel Evaluation).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All tensor pointers are DEVICE pointers owned by the caller.  The
 *   library never allocates device memory; scratch space is passed in as a
 *   caller-owned workspace whose size the *_workspace_bytes functions give
 *   (bpc_decode_attention_noalloc instead uses a static array the library
 *   holds on each GPU, see there).
 * - bf16 tensors are passed as `const uint16_t*` bit patterns.
 * - Strides are in elements of the pointed-to type; the innermost
 *   dimension (D for K, V, q, P; the W code words of one key) is contiguous.
 * - Shapes: B sequences, Hq query heads, Hkv KV heads (Hq = G Hkv with the
 *   group size G in {1, 2, 4, 8, 16}; query head j reads KV head j / G),
 *   N cached keys, D = 128 head dim,
 *   L in {32, 64, 128} code bits, W = L / 32 words per code.
 * - Code bit i of a key is bit (i % 32) of 32-bit word i / 32; a set bit
 *   means h_i = +1.
 * - Calls are asynchronous on `stream` (a hipStream_t; NULL = the default
 *   stream).  All argument checks happen on the host before anything is
 *   enqueued: on error nothing is launched and no output is touched.
 *   Faults during kernel execution surface at the caller's next sync.
 * - Pointers must be 16-byte aligned and row strides multiples of 8
 *   elements (16 bytes), else BPC_EALIGN.
 * - Calls share no mutable state except a thread-local error message (and,
 *   for bpc_decode_attention_noalloc, that GPU's static scratch), so they
 *   are reentrant; two calls that share an output or a workspace must not
 *   overlap in time.
 * - Arithmetic that decides a code bit is IEEE binary64 in a fixed order:
 *   dot products over D split D into 4 consecutive blocks of D/4, sum each
 *   block in ascending order from +0 with separately rounded multiplies and
 *   adds, and combine them as ((b0 + b1) + (b2 + b3)); sums over N rows use
 *   the pairwise tree (adjacent pairs, odd last element carried);
 *   sign(a) = +1 iff a >= 0.  A sign decision is counted as "fragile" when
 *   |(float)a| < 1e-6.
 */
#ifndef BPC_H
#define BPC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes (0 = success). */
#define BPC_OK 0
#define BPC_EINVAL (-1)       /* null required pointer, bad size or shape */
#define BPC_EUNSUPPORTED (-2) /* D != 128 or L not in {32, 64, 128} */
#define BPC_EALIGN (-3)       /* pointer or row stride not 16-byte aligned */
#define BPC_EWORKSPACE (-4)   /* workspace missing or too small */
#define BPC_EHIP (-5)         /* a HIP runtime call or launch failed */

/* Static description of a status code. */
const char* bpc_status_string(int status);

/* Detail of the last failed call on the calling thread ("" if none). */
const char* bpc_last_error(void);

/* Library version, major * 10000 + minor * 100 + patch. */
int bpc_version(void);

/*
 * bpc_set_decode_path -- how the decode entry points run a step, for this
 * process: 0 (the default) runs it as one fused launch whenever every
 * workgroup of the step fits on the current device at once, else as three
 * launches; the fused launch splits each (b, h) into slices of 16384 keys,
 * or of 4096 or 8192 keys (code lengths 32 and 64, groups of up to 8 query
 * heads) when those still fit, at most two workgroups per compute unit, and
 * the larger slices would leave most of the device idle.  1 always uses the three
 * launches, 2 the fused launch on 16384-key slices only (both for
 * comparisons and tests).  Calls already enqueued are not affected;
 * workspace sizes follow the path (bpc_decode_workspace_bytes queries it).
 * Returns BPC_EINVAL for any other value.
 */
int bpc_set_decode_path(int path);

/*
 * bpc_decode_slice_keys -- keys per slice (16384, 8192 or 4096) a decode step of
 * this shape would use on the current device under the current setting (the
 * three-launch path always uses 16384); shapes the decode entry points
 * reject return 0.
 */
int bpc_decode_slice_keys(int B, int Hq, int Hkv, int N, int L);

/*
 * bpc_decode_path_taken -- which path a decode step of this shape would take
 * on the current device under the current bpc_set_decode_path setting:
 * 0 = one fused launch, 1 = three launches.  Queries the device's occupancy
 * (the first query per device and kernel instance); shapes the decode entry
 * points reject return 1.
 */
int bpc_decode_path_taken(int B, int Hq, int Hkv, int N, int L);

/*
 * bpc_build_hash -- binary principal components of each (sequence, KV
 * head)'s keys (Sec. 3.2, "Binary Principal Components Finding", Algorithm
 * "Constructing hash codes and corresponding hashing projection"; the
 * closed-form v for a fixed u is in the Appendix "Procedure Overview").
 *
 * For every (b, h) independently, with residual R = K[b,h,0:N,:] and for
 * i = 0..L-1:
 *     a_j = R_j . G[i]           (fixed-order fp64 dot, see above)
 *     u_j = sign(a_j)            code bit i of key j
 *     v   = (sum_j u_j R_j) / N  (pairwise tree over j, one rounded divide)
 *     P[i] = (float)v
 *     R_j = R_j - u_j P[i]       (the stored float P is what is removed)
 * G [L, D] fp32 holds the random Gaussian directions (v* of the
 * algorithm), supplied by the caller and shared by all (b, h).
 *
 * K         [B, Hkv, >=N, D] bf16, strides sK_b, sK_h, sK_n (elements)
 * G         [L, D] fp32, contiguous
 * P_out     [B, Hkv, L, D] fp32, contiguous (written)
 * codes_out [B, Hkv, >=N, W] uint32, strides sC_b, sC_h (words); key rows
 *           are W words apart (written)
 * err_out   [B, Hkv, N] fp32 contiguous, ||k_j - h_j P|| (or NULL)
 * fragile_out  one device uint64 to which the number of fragile sign
 *           decisions is ADDED (the caller zeroes it), or NULL
 * workspace    device memory of at least bpc_build_workspace_bytes(...)
 *           bytes, 256-byte aligned; its contents on entry do not matter.
 * Cost: 2 L + 2 kernel launches.  With that workspace nothing of size N x D
 * is stored: each bit's pass recomputes R_j from the bf16 key, the key's
 * code bits so far and P (the same rounded subtractions, in the same
 * order), so the workspace holds one fp64 partial sum per 128-key chunk
 * and coordinate plus fp64 copies of P and G.  Given at least
 * bpc_build_checkpoint_workspace_bytes(...) bytes (1 KiB more per key,
 * rounded up to 128-key chunks), the build also keeps each key's fp64
 * residual there every 16 bits and later passes start from it, trading
 * that memory and its traffic for fewer recomputed subtractions; the
 * results are bit for bit the same.
 */
size_t bpc_build_workspace_bytes(int B, int Hkv, int N, int D, int L);
size_t bpc_build_checkpoint_workspace_bytes(int B, int Hkv, int N, int D, int L);
int bpc_build_hash(const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                   int B, int Hkv, int N, int D, int L,
                   const float* G,
                   float* P_out,
                   uint32_t* codes_out, int64_t sC_b, int64_t sC_h,
                   float* err_out,
                   unsigned long long* fragile_out,
                   void* workspace, size_t workspace_bytes,
                   void* stream);

/*
 * bpc_hash_keys -- hash keys against a given projection (Sec. 3.2,
 * Algorithm "Given projection, computing hashcode"; also the per-key
 * "hashing kernel" of the Appendix "CUDA Optimizations on Bitwise
 * Operations").  Per key: r = k; for i = 0..L-1: u = sign(r . P[i]);
 * r = r - u P[i]; h_i = u.
 *
 * K          [B, Hkv, >=N, D] bf16, strides sK_b, sK_h, sK_n
 * P          [B, Hkv, L, D] fp32 with strides sP_b, sP_h (elements; rows of
 *            one head are contiguous).  sP_b = sP_h = 0 shares one P.
 * codes_out  [B, Hkv, >=N, W] uint32, strides sC_b, sC_h (written)
 * err_out    [B, Hkv, N] fp32 contiguous ||r_final|| (or NULL)
 * fragile_out  device uint64 accumulator (or NULL), as above.
 * No workspace; one kernel launch.
 */
int bpc_hash_keys(const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                  int B, int Hkv, int N, int D, int L,
                  const float* P, int64_t sP_b, int64_t sP_h,
                  uint32_t* codes_out, int64_t sC_b, int64_t sC_h,
                  float* err_out,
                  unsigned long long* fragile_out,
                  void* stream);

/*
 * bpc_hash_keys_mm -- the codes of bpc_hash_keys, bit for bit, and the same
 * fragile count, with the projections on the matrix cores (Algorithm "Given
 * projection, computing hashcode"; App. "CUDA Optimizations on Bitwise
 * Operations", hashing kernel).  Unrolling the residual of Algorithm 2
 * gives a_i = k . P_i - sum_{t<i} u_t (P_t . P_i): the products k . P_i are
 * one dense contraction (bf16 MFMA on P cut exactly into three bf16 parts,
 * fp32 accumulation), the sum over earlier bits uses the Gram matrix of P in
 * fp32.  Each sign is kept only when |a^| exceeds a bound on its distance to
 * the fixed-order fp64 value of bpc_hash_keys (plus the fragile threshold);
 * every other decision is recomputed in that fixed-order arithmetic.
 *
 * Arguments as for bpc_hash_keys, without err_out (residual norms need the
 * fp64 residual itself: use bpc_hash_keys for them).
 * fallbacks_out  device uint64 accumulator (or NULL): decisions recomputed
 *            in the fixed-order arithmetic.
 * No workspace; one kernel launch.
 */
int bpc_hash_keys_mm(const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                     int B, int Hkv, int N, int D, int L,
                     const float* P, int64_t sP_b, int64_t sP_h,
                     uint32_t* codes_out, int64_t sC_b, int64_t sC_h,
                     unsigned long long* fragile_out,
                     unsigned long long* fallbacks_out,
                     void* stream);

/*
 * bpc_append_kv -- decode-time append of T new tokens to the cache: their
 * key and value rows are stored at positions [pos, pos + T) of K and V, and
 * each new key is hashed against the given projection with the iterative
 * residual of Algorithm "Given projection, computing hashcode" (Sec. 3.2:
 * the setting "where the projection matrix P is given"), its code stored at
 * the same positions of `codes`.  The arithmetic and the code bits are those
 * of bpc_hash_keys.  P stays fixed, as the paper's decode phase keeps it.
 *
 * k_new, v_new [B, Hkv, T, D] bf16, strides (sKn_b, sKn_h, sKn_t) and
 *            (sVn_b, sVn_h, sVn_t)
 * K, V       [B, Hkv, Ncap, D] bf16 caches, strides as in bpc_decode_attention
 *            (rows pos .. pos + T - 1 written)
 * codes      [B, Hkv, Ncap, W] uint32, strides sC_b, sC_h (rows written)
 * P          [B, Hkv, L, D] fp32, strides sP_b, sP_h (0, 0 = shared)
 * Ncap       rows the caches hold; 0 <= pos and pos + T <= Ncap
 * err_out    [B, Hkv, T] fp32 contiguous ||k - h P|| of the new keys (or NULL)
 * fragile_out  device uint64 accumulator (or NULL), as for bpc_hash_keys.
 * No workspace; one kernel launch.
 */
int bpc_append_kv(const uint16_t* k_new, int64_t sKn_b, int64_t sKn_h, int64_t sKn_t,
                  const uint16_t* v_new, int64_t sVn_b, int64_t sVn_h, int64_t sVn_t,
                  uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                  uint16_t* V, int64_t sV_b, int64_t sV_h, int64_t sV_n,
                  uint32_t* codes, int64_t sC_b, int64_t sC_h,
                  const float* P, int64_t sP_b, int64_t sP_h,
                  int B, int Hkv, int Ncap, int pos, int T, int D, int L,
                  float* err_out,
                  unsigned long long* fragile_out,
                  void* stream);

/*
 * bpc_decode_attention -- one decode step of BinaryPC sparse attention
 * (Sec. 3.2 "Retrieval Phase"; Algorithm "Computing hashing score";
 * Sec. 4.2 "Kernel Evaluation": search, selection, gathering, attention).
 *
 * For every (b, KV head h) with its group of G = Hq / Hkv query heads:
 *  1. x = sum_g q_g P^T (fixed-order fp64 dots, heads added in ascending
 *     order); m = max |x_i|; p_i = round-half-away((x_i * 127) / m) in
 *     [-127, 127] (p = 0 if m = 0).  Packed as 8 planes of W words: plane 0
 *     bit i = (p_i >= 0), plane 1 + j bit i = bit j of |p_i|.
 *  2. score of cached key n: c_n = sum_i h_{n,i} p_i, computed as
 *     sum|p| - 2 * sum_j 2^j popcount(plane_{1+j} & (code_n XOR plane_0)).
 *  3. the k keys with the largest c (equal scores: lower index first).
 *  4. out[b, g] = softmax over the selected n of (q_g . K_n) * sm_scale,
 *     applied to V_n; fp32 accumulation.
 *
 * q          [B, Hq, D] bf16, contiguous
 * K, V       [B, Hkv, >=N, D] bf16, strides (sK_b, sK_h, sK_n) and
 *            (sV_b, sV_h, sV_n)
 * codes      [B, Hkv, >=N, W] uint32, strides sC_b, sC_h
 * P          [B, Hkv, L, D] fp32, strides sP_b, sP_h (0, 0 = shared)
 * N          1 <= N <= 16777216 cached keys per (b, KV head)
 * k          1 <= k <= N selected keys per (b, KV head)
 * out        [B, Hq, D] fp32, contiguous (written)
 * idx_out    [B, Hkv, k] int32 selected key indices, ascending (or NULL)
 * score_out  [B, Hkv, N] int32 scores c_n (or NULL)
 * qcode_out  [B, Hkv, 8, W] uint32 packed query planes (or NULL)
 * workspace  at least bpc_decode_workspace_bytes(...) bytes, 256-byte
 *            aligned.  Its first 1088 KiB (BPC_DECODE_ZEROED_BYTES) must be
 *            zero before the first call on it (allocate it zeroed); every
 *            call leaves them zero.  The rest may hold anything.  Two calls
 *            that use the same workspace must be ordered on one stream.
 *            The size depends on the path the current device takes (below).
 * Cost: when every workgroup of the step fits on the device at once (a
 * slice of 16384 keys per workgroup; e.g. 1024 slices at L = 64 and G <= 4
 * on MI355X), one fused launch: each slice is packed and scored, the slices
 * of a (b, h) exchange their histogram summaries through the workspace,
 * select, gather and attend, and the last slice of (b, h) merges the
 * partials.  Otherwise three launches (query packing with scoring, threshold
 * with selection and attention, merge of the per-slice partials), plus one
 * for a ragged last slice or codes whose strides are not multiples of 4
 * words.  bpc_set_decode_path selects the three launches for comparisons.
 */
#define BPC_DECODE_ZEROED_BYTES (1088u * 1024u)
size_t bpc_decode_workspace_bytes(int B, int Hq, int Hkv, int N, int D, int L, int k);
int bpc_decode_attention(const uint16_t* q,
                         const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                         const uint16_t* V, int64_t sV_b, int64_t sV_h, int64_t sV_n,
                         const uint32_t* codes, int64_t sC_b, int64_t sC_h,
                         const float* P, int64_t sP_b, int64_t sP_h,
                         int B, int Hq, int Hkv, int N, int D, int L, int k,
                         float sm_scale,
                         float* out,
                         int32_t* idx_out,
                         int32_t* score_out,
                         uint32_t* qcode_out,
                         void* workspace, size_t workspace_bytes,
                         void* stream);

/*
 * bpc_decode_attention_per_head -- the decode step with one selection per
 * QUERY head instead of one per KV head (the alternative to the group rule
 * of bpc_decode_attention; Sec. 3.2 "Retrieval Phase", Alg. 3, App. A.3
 * "Scoring kernel", which scores query-key pairs head by head): query head j
 * projects and quantises its own q_j P^T, scores every cached code of KV
 * head floor(j / G) against it, takes its own top-k (ties to the lower
 * index) and attends over its own selection.
 *
 * Arguments as for bpc_decode_attention, except:
 * idx_out    [B, Hq, k] int32, ascending per query head (or NULL)
 * score_out  [B, Hq, N] int32 (or NULL)
 * qcode_out  [B, Hq, 8, L/32] uint32 (or NULL)
 * workspace  at least bpc_decode_per_head_workspace_bytes(...) bytes,
 *            256-byte aligned.
 * Any power-of-two or other group size G = Hq / Hkv is accepted.
 * Cost: the codes of a KV head are scanned once per query head (G times
 * the code traffic of bpc_decode_attention) and G selections are gathered.
 * When the batch stride of K, V, codes and P is Hkv times the head stride
 * (contiguous heads) the batch is one launch sequence of three kernels;
 * otherwise one per sequence.  Errors as for bpc_decode_attention.
 */
size_t bpc_decode_per_head_workspace_bytes(int B, int Hq, int Hkv, int N, int D, int L, int k);
int bpc_decode_attention_per_head(const uint16_t* q,
                                  const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                                  const uint16_t* V, int64_t sV_b, int64_t sV_h, int64_t sV_n,
                                  const uint32_t* codes, int64_t sC_b, int64_t sC_h,
                                  const float* P, int64_t sP_b, int64_t sP_h,
                                  int B, int Hq, int Hkv, int N, int D, int L, int k,
                                  float sm_scale,
                                  float* out,
                                  int32_t* idx_out,
                                  int32_t* score_out,
                                  uint32_t* qcode_out,
                                  void* workspace, size_t workspace_bytes,
                                  void* stream);

/*
 * bpc_select_hard -- the hard-to-hash set of the Error-Aware Safeguard
 * (Sec. 3.2 "Error-Aware Safeguard (EAS)", Eq. reconstruction_error): for
 * every (b, KV head), the m keys with the largest reconstruction errors
 * ||k - h P|| (the err_out of bpc_build_hash or bpc_hash_keys).  Errors are
 * compared in the IEEE total order of float32; equal errors go to the lower
 * index.
 *
 * err       [B, Hkv, N] fp32, strides sE_b, sE_h (elements), keys contiguous
 * m         0 <= m <= N (m = 0: nothing is written)
 * serr_out  [B, Hkv, m] int32, contiguous: the selected key indices in
 *           ascending order (written)
 * Both pointers 4-byte aligned.  No workspace; one kernel launch (one
 * workgroup per (b, KV head) making four passes over its N errors).
 */
int bpc_select_hard(const float* err, int64_t sE_b, int64_t sE_h, int B, int Hkv, int N, int m,
                    int32_t* serr_out, void* stream);

/*
 * bpc_decode_attention_eas -- bpc_decode_attention with the Error-Aware
 * Safeguard (Sec. 3.2, Eq. safeguard_union): attention runs over
 * S_attn = S_hash u S_err, where S_hash are the k keys with the highest hash
 * scores (selected exactly as by bpc_decode_attention) and S_err is the
 * caller's hard-to-hash set (from bpc_select_hard at prefill).  The paper
 * reserves 10 % of the token budget for S_err: with a budget of n keys the
 * caller passes m = ceil(n / 10) hard keys and k = n - m.  |S_attn| is
 * between k and k + m.
 *
 * serr      [B, Hkv, m] int32 with strides sS_b, sS_h: per (b, h) distinct
 *           key indices in [0, N) in ascending order (bpc_select_hard's
 *           output has this form; entries outside [0, N) are ignored)
 * m         0 <= m <= N; m = 0 is bpc_decode_attention
 * idx_out   [B, Hkv, k] int32: S_hash, ascending (or NULL)
 * added_out [B, Hkv, m] int32 contiguous: 1 where the entry of S_err was
 *           not in S_hash and was added, 0 where it was already selected
 *           (or NULL)
 * All other arguments, the workspace size and the error behaviour are those
 * of bpc_decode_attention.
 */
int bpc_decode_attention_eas(const uint16_t* q,
                             const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                             const uint16_t* V, int64_t sV_b, int64_t sV_h, int64_t sV_n,
                             const uint32_t* codes, int64_t sC_b, int64_t sC_h,
                             const float* P, int64_t sP_b, int64_t sP_h,
                             int B, int Hq, int Hkv, int N, int D, int L, int k,
                             float sm_scale,
                             const int32_t* serr, int64_t sS_b, int64_t sS_h, int m,
                             float* out,
                             int32_t* idx_out,
                             int32_t* added_out,
                             void* workspace, size_t workspace_bytes,
                             void* stream);

/*
 * bpc_dense_attention -- dense decode attention over all N cached keys
 * (softmax of (q_g . K_n) * sm_scale over n = 0..N-1, applied to V; fp32
 * accumulation).  Not part of the method: it is the comparison point the
 * paper's efficiency results are quoted against (full attention at decode,
 * Sec. 4.2 "Efficiency Evaluation"), provided for measuring the sparse step
 * against.  Arguments as for bpc_decode_attention; the workspace holds the
 * per-chunk partials, bpc_dense_workspace_bytes(...) bytes, 256-byte aligned.
 * Cost: two kernel launches.
 */
size_t bpc_dense_workspace_bytes(int B, int Hq, int Hkv, int N, int D);
int bpc_dense_attention(const uint16_t* q,
                        const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                        const uint16_t* V, int64_t sV_b, int64_t sV_h, int64_t sV_n,
                        int B, int Hq, int Hkv, int N, int D,
                        float sm_scale,
                        float* out,
                        void* workspace, size_t workspace_bytes,
                        void* stream);

/*
 * bpc_decode_attention_profiled -- bpc_decode_attention that also records
 * caller-created hipEvent_t handles on `stream` at the stage boundaries
 * (query packing and scoring | threshold, selection and attention | merge):
 * events[0] before the first stage and events[s + 1] after stage s, so
 * n_events must be BPC_DECODE_STAGES + 1.  For measuring only.
 */
#define BPC_DECODE_STAGES 3
int bpc_decode_attention_profiled(const uint16_t* q,
                                  const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                                  const uint16_t* V, int64_t sV_b, int64_t sV_h, int64_t sV_n,
                                  const uint32_t* codes, int64_t sC_b, int64_t sC_h,
                                  const float* P, int64_t sP_b, int64_t sP_h,
                                  int B, int Hq, int Hkv, int N, int D, int L, int k,
                                  float sm_scale,
                                  float* out,
                                  int32_t* idx_out,
                                  int32_t* score_out,
                                  uint32_t* qcode_out,
                                  void* workspace, size_t workspace_bytes,
                                  void* stream,
                                  void* const* events, int n_events);

/*
 * bpc_decode_attention_noalloc -- bpc_decode_attention for callers that
 * cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): the same computation and
 * kernels, with the workspace taken from a static device array inside the
 * library instead of a caller argument.  The call itself allocates nothing.
 *
 * Arguments, outputs and errors as for bpc_decode_attention, without the
 * workspace arguments.  `stream` must belong to the current device.
 * Limit: the decode workspace of the call (bpc_decode_workspace_bytes) must
 * fit the array, bpc_decode_noalloc_max_bytes() = 64 MiB; a larger call
 * returns BPC_EWORKSPACE and launches nothing.  (The fused single-launch
 * path needs about 5 MiB at batch 16 x 8 KV heads x 131072 keys; the
 * three-launch path, taken when a step's workgroups do not all fit on the
 * GPU at once, needs about 100 KiB per 16384-key slice, so 64 MiB covers
 * about 640 slices of it.)
 * Each GPU holds one such array for the life of the process, and every call
 * on that GPU uses it: two calls on one GPU that overlap in time (different
 * streams without ordering, different host threads) race on it and give
 * undefined results.  Calls ordered on one stream are safe.  Nothing in the
 * array has to hold a particular value when a call starts.
 */
size_t bpc_decode_noalloc_max_bytes(void);
int bpc_decode_attention_noalloc(const uint16_t* q,
                                 const uint16_t* K, int64_t sK_b, int64_t sK_h, int64_t sK_n,
                                 const uint16_t* V, int64_t sV_b, int64_t sV_h, int64_t sV_n,
                                 const uint32_t* codes, int64_t sC_b, int64_t sC_h,
                                 const float* P, int64_t sP_b, int64_t sP_h,
                                 int B, int Hq, int Hkv, int N, int D, int L, int k,
                                 float sm_scale,
                                 float* out,
                                 int32_t* idx_out,
                                 int32_t* score_out,
                                 uint32_t* qcode_out,
                                 void* stream);

#ifdef __cplusplus
}
#endif

#endif /* BPC_H */
