/*
 * bd_attn — block-diffusion masked attention (forward and backward) for
 * AMD Instinct MI355X (gfx950).
 *
 * The operation (DiRL, arXiv 2512.22234, Section 4.1 with the block rules of
 * Section 2.1, Eq. 1 and Eq. 2): attention over a packed sequence of 2L
 * tokens [x_t | x_0], the noisy copy first.  With the block index
 * b(p) = (p mod L) div S of packed position p:
 *   - a noisy query (p < L) sees noisy keys of its own block (both
 *     directions) and clean keys of strictly earlier blocks;
 *   - a clean query sees clean keys of its own and earlier blocks and never
 *     a noisy key.
 * O = softmax(scale * Q K^T restricted to visible keys) V, per query head h,
 * using KV head h div (Hq / Hkv).
 *
 * Layouts (all contiguous, innermost dimension last, 16-byte aligned):
 *   Q, O, dO, dQ : [B, Hq,  2L, D]
 *   K, V, dK, dV : [B, Hkv, 2L, D]
 *   LSE          : [B, Hq,  2L] float32 (4-byte aligned), natural-log
 *                  log-sum-exp of the scaled scores of each row over its
 *                  visible keys.
 * Element type of Q/K/V/O/dO/dQ/dK/dV is selected by `dtype`:
 *   BD_ATTN_BF16 (0): bfloat16 — the compute path;
 *   BD_ATTN_FP32 (1): a float32 interface to the bfloat16 path, not float32
 *                     arithmetic.  Inputs are rounded to bfloat16 (nearest
 *                     even) inside the library, every product runs on the
 *                     bf16 MFMAs with float32 accumulation, and the bf16
 *                     results are widened to float32.  The accuracy is that
 *                     of bfloat16 inputs: for unit-variance inputs at D = 64
 *                     the rounding alone moves LSE by up to ~3e-3 and O by
 *                     ~2.5e-3 relative (L2), exact arithmetic on both sides.
 * D must be 64 or 128; 1 <= L <= 2^22.  S >= L behaves as S = L.  S need
 * not divide L (the last block is then shorter).  scale <= 0 selects
 * 1/sqrt(D).
 *
 * Ownership and ordering: the caller allocates every buffer, including the
 * workspace (size from bd_attn_workspace_bytes, at least 16-byte aligned).  The
 * library never allocates, frees or synchronises; all work is enqueued on
 * `stream` in order and the call returns without waiting.  Outputs must not
 * overlap inputs.  The workspace may be reused once the enqueued work has
 * completed (stream order guarantees this for calls on the same stream).
 * Apart from the scratch array of bd_attn_bwd_noalloc (and the per-device
 * address of it, looked up once under a lock), the library keeps no mutable
 * global state; calls from several host threads are safe.
 *
 * Errors: every entry point validates its arguments before enqueuing
 * anything; a call that returns non-zero has enqueued no work (except
 * BD_ATTN_ERR_HIP, reported from the launch itself).  No C++ exception
 * crosses this interface.
 */
#ifndef BD_ATTN_H
#define BD_ATTN_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum bd_attn_status {
  BD_ATTN_OK = 0,
  BD_ATTN_ERR_INVALID_ARGUMENT = 1, /* null/misaligned pointer, B,L,S<1, L>2^22, Hq%Hkv!=0, overlap */
  BD_ATTN_ERR_UNSUPPORTED = 2,      /* D not in {64,128}, unknown dtype */
  BD_ATTN_ERR_WORKSPACE_TOO_SMALL = 3, /* checked before overlap with the workspace */
  BD_ATTN_ERR_HIP = 4,              /* a HIP launch reported an error */
  BD_ATTN_ERR_EXCEEDS_SCRATCH = 5   /* bd_attn_bwd_noalloc: the problem needs more than its scratch */
};

enum bd_attn_dtype { BD_ATTN_BF16 = 0, BD_ATTN_FP32 = 1 };

/* Tile classes returned by bd_attn_classify_tiles_host. */
enum bd_attn_tile_class { BD_TILE_EMPTY = 0, BD_TILE_FULL = 1, BD_TILE_PARTIAL = 2 };

/*
 * Forward pass (Section 4.1; masking rules of Eq. 1 and Eq. 2).
 * Inputs Q, K, V; outputs O (same dtype as the inputs) and LSE (float32).
 * ws/ws_bytes: device workspace of at least
 * bd_attn_workspace_bytes(B, L, S, Hq, Hkv, D, dtype, 0) bytes (zero for
 * bfloat16 inputs; ws may then be NULL).
 */
int bd_attn_fwd(const void* Q, const void* K, const void* V,
                int B, int L, int S, int Hq, int Hkv, int D, float scale, int dtype,
                void* O, float* LSE, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Backward pass: the vector-Jacobian product of the forward pass for the
 * upstream gradient dO, given the forward's O and LSE.  Writes dQ, dK, dV
 * (dK and dV summed over the Hq/Hkv query heads sharing each KV head).
 * Deterministic: no floating-point atomics, so results are bitwise
 * reproducible.  The only atomics are integer counters per group of 32 keys
 * of each clean key tile (arrivals and published parts), with which the
 * workgroups that split that tile's query walk (two, or four for shapes with
 * few KV heads x length) decide which of them adds the others' float32 sums;
 * the sums are added in part order, so the result is the same whichever part
 * finishes last.  Should that meeting ever fail to complete within its
 * bounded wait, the affected dK/dV rows are written as NaN rather than as a
 * partial sum.
 * ws/ws_bytes: at least bd_attn_workspace_bytes(..., for_bwd = 1) bytes.
 */
int bd_attn_bwd(const void* dO, const void* Q, const void* K, const void* V,
                const void* O, const float* LSE,
                int B, int L, int S, int Hq, int Hkv, int D, float scale, int dtype,
                void* dQ, void* dK, void* dV, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * bd_attn_bwd without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation).  Same arguments, work, results (bitwise) and
 * validation as bd_attn_bwd; the workspace is a fixed device array inside the
 * library of BD_ATTN_NOALLOC_SCRATCH_BYTES bytes, one per GPU, held from the
 * library's first use on that GPU until the process ends.  A problem whose
 * bd_attn_workspace_bytes(..., for_bwd = 1) exceeds it is rejected with
 * BD_ATTN_ERR_EXCEEDS_SCRATCH before anything is enqueued (in bfloat16 the
 * workspace is B*Hq*2L*8 + (n-1)*B*Hkv*L'*D*8 bytes plus a few KiB (L' = L rounded
 * up to a multiple of 128), where n is
 * the number of parts each clean key tile's dK/dV walk is split into: 4 when
 * B*Hkv*(L+128) <= 21845, else 2; 34.0 MiB for B=2, Hq=32, Hkv=8, D=128,
 * L=2048 and 68.0 MiB for B=1, L=8192 at the same heads; float32 inputs also
 * need bf16 copies of every tensor).  The call
 * allocates and frees nothing; its first call on a GPU looks up that GPU's
 * copy of the array.  All calls on one GPU share the array and leave their
 * contents in it: calls whose work may overlap in time on one GPU (other
 * streams, other host threads) race and must be serialised by the caller.
 */
#define BD_ATTN_NOALLOC_SCRATCH_BYTES ((size_t)96 << 20)
int bd_attn_bwd_noalloc(const void* dO, const void* Q, const void* K, const void* V,
                        const void* O, const float* LSE,
                        int B, int L, int S, int Hq, int Hkv, int D, float scale, int dtype,
                        void* dQ, void* dK, void* dV, hipStream_t stream);

/*
 * Workspace bytes needed by bd_attn_fwd (for_bwd = 0) or bd_attn_bwd
 * (for_bwd = 1).  Returns 0 for arguments the calls would reject.
 */
size_t bd_attn_workspace_bytes(int B, int L, int S, int Hq, int Hkv, int D, int dtype, int for_bwd);

/*
 * Host-side copy of the tile classifier the kernels use (exposed for tests).
 * Tiles are half-local: each half of the packed sequence is cut into
 * ceil(L/BM) query tiles and ceil(L/BN) key tiles, the last one shorter when
 * L is not a multiple; no tile straddles position L.  Writes one class per
 * (query tile, key tile) pair, row-major, into out[nq * nk] with
 * nq = 2*ceil(L/BM), nk = 2*ceil(L/BN) (query tiles and key tiles numbered
 * noisy half first).  EMPTY: no visible pair; FULL: every pair visible and
 * both tiles full-sized; PARTIAL otherwise.  Returns a status.
 */
int bd_attn_classify_tiles_host(int L, int S, int BM, int BN, int8_t* out);

/*
 * Host-side copy of the tile walk the kernels perform (exposed for tests).
 * Same tiling and out[] indexing as bd_attn_classify_tiles_host; writes, per
 * (query tile, key tile) pair, how many times the kernels visit it: walking
 * key tiles per query tile (forward and dQ, by_key_tile = 0) or query tiles
 * per key tile (dK/dV, by_key_tile = 1; that kernel repeats the walk for each
 * query head of the group, and splits each clean key tile's walk into nsplit
 * parts, 2 or 4; nsplit is ignored for by_key_tile = 0, and any other value
 * with by_key_tile = 1 is BD_ATTN_ERR_INVALID_ARGUMENT).  A correct walk visits every non-EMPTY pair
 * exactly once.  A visited pair whose class, as the kernels compute it
 * without divisions (and the two-comparison FULL test the kernels apply
 * per step), differs from bd_attn_classify_tiles_host's gets 64 instead
 * of 1; so does a key tile that the forward and dQ kernels would run in
 * their leading loop of FULL tiles (no visibility test) without it being
 * FULL.
 */
int bd_attn_visit_lists_host(int L, int S, int BM, int BN, int by_key_tile, int nsplit, int8_t* out);

/*
 * Host-side copy of the per-element visibility rule of PARTIAL tiles
 * (exposed for tests): the kernels test a position against a window
 * [lo, hi) computed once per row.  Writes the 2L x 2L mask out[q*2L + k]
 * (1 = visible) rebuilt from the windows of every query row (by_key = 0,
 * forward and dQ) or of every key row (by_key = 1, dK/dV).
 */
int bd_attn_mask_windows_host(int L, int S, int by_key, int8_t* out);

/*
 * Tests only: the visibility windows of runs of `group` consecutive positions
 * of one half (the runs start at multiples of `group`; the last one of a half
 * may be shorter), i.e. the union over the run's rows of the windows above,
 * expanded into the same 2L x 2L layout: out[q * 2L + k] = 1 iff key k is
 * visible from some query of q's run (by_key = 0), or some key of k's run is
 * visible from query q (by_key = 1).  The kernels skip, per wave, the 32-key
 * or 32-query blocks outside the window of the wave's own 32-row run.
 * Returns BD_ATTN_ERR_INVALID_ARGUMENT for L, S or group < 1 or a null `out`.
 */
int bd_attn_group_windows_host(int L, int S, int by_key, int group, int8_t* out);

/*
 * Benchmark variants of bd_attn_fwd / bd_attn_bwd: identical work and
 * validation, and in addition caller-created events recorded from the kernel
 * dispatches themselves (hipExtLaunchKernelGGL): kernel launch i records
 * marks[2i] as it begins and marks[2i + 1] as it ends, for as many launches
 * as n_marks covers (n_marks = 2 x the launches for all of them).  The
 * events put no packet of their own in the stream, so the kernels follow
 * each other as in the plain calls.  The kernels launched, in order, are
 * named by bd_attn_stage_names.  Intended for measuring each kernel's
 * duration on the stream it runs on.
 */
int bd_attn_fwd_marked(const void* Q, const void* K, const void* V,
                       int B, int L, int S, int Hq, int Hkv, int D, float scale, int dtype,
                       void* O, float* LSE, void* ws, size_t ws_bytes, hipStream_t stream,
                       hipEvent_t* marks, int n_marks);
int bd_attn_bwd_marked(const void* dO, const void* Q, const void* K, const void* V,
                       const void* O, const float* LSE,
                       int B, int L, int S, int Hq, int Hkv, int D, float scale, int dtype,
                       void* dQ, void* dK, void* dV, void* ws, size_t ws_bytes, hipStream_t stream,
                       hipEvent_t* marks, int n_marks);

/*
 * Packed sequences ("dynamic packing", named in Section 5.2 as the next
 * speed-up of blockwise training): n_seqs sequences of different lengths in
 * one buffer, each a [x_t | x_0] pair with the mask of Section 4.1 (Eq. 1 and
 * Eq. 2 at the sequence's own positions); sequences never attend to each
 * other.
 *
 * cu_seqlens: DEVICE array of n_seqs + 1 int32 values (4-byte aligned),
 *   cu_seqlens[0] = 0, non-decreasing, cu_seqlens[n_seqs] = total_L; sequence
 *   i has L_i = cu_seqlens[i+1] - cu_seqlens[i] tokens per copy (0 allowed).
 *   It is read by the kernels only, not by the host.
 * max_L: an upper bound on every L_i (it sizes the launch grids); 1 <= max_L
 *   <= 2^22.  A sequence longer than max_L is only partly computed: the caller
 *   must pass a true bound.
 * Layouts (contiguous, innermost last): Q, O, dO, dQ [Hq, 2*total_L, D];
 *   K, V, dK, dV [Hkv, 2*total_L, D]; LSE [Hq, 2*total_L].  Sequence i occupies
 *   rows [2*cu_seqlens[i], 2*cu_seqlens[i+1]) of every head: its noisy copy,
 *   then its clean copy.
 * S: block size, the same for every sequence (a sequence shorter than S is
 *   one block).  Everything else (dtype, scale, workspace, ownership, stream
 *   order, errors, determinism) is as for bd_attn_fwd / bd_attn_bwd; with
 *   total_L = 0 the calls validate and enqueue nothing.
 */
int bd_attn_varlen_fwd(const void* Q, const void* K, const void* V, const int32_t* cu_seqlens, int n_seqs,
                       int total_L, int max_L, int S, int Hq, int Hkv, int D, float scale, int dtype,
                       void* O, float* LSE, void* ws, size_t ws_bytes, hipStream_t stream);
int bd_attn_varlen_bwd(const void* dO, const void* Q, const void* K, const void* V, const void* O,
                       const float* LSE, const int32_t* cu_seqlens, int n_seqs, int total_L, int max_L,
                       int S, int Hq, int Hkv, int D, float scale, int dtype,
                       void* dQ, void* dK, void* dV, void* ws, size_t ws_bytes, hipStream_t stream);
/* Workspace bytes for bd_attn_varlen_fwd (for_bwd = 0) or bd_attn_varlen_bwd
 * (for_bwd = 1); 0 for arguments the calls would reject. */
size_t bd_attn_varlen_workspace_bytes(int n_seqs, int total_L, int max_L, int S, int Hq, int Hkv, int D,
                                      int dtype, int for_bwd);

/*
 * Block decoding over a KV cache (Section 2.1: blockwise models keep the
 * K/V of finished blocks in a cache; the block being denoised attends to
 * that cache and, in both directions, to itself, Eq. 2).  For each sequence
 * b and query head h, the S noisy queries of the current block attend to the
 * first cache_lens[b] rows of the KV head's cache followed by the block's
 * own S keys, with no further mask: the noisy rows of the training mask of
 * Section 4.1 for a block whose earlier blocks are all cached.
 *
 * Layouts (contiguous, innermost last, bfloat16, 16-byte aligned):
 *   Q, O             : [B, Hq, S, D]
 *   K_cache, V_cache : [B, Hkv, capacity, D]   (rows past cache_lens[b] are not read)
 *   K_new, V_new     : [B, Hkv, S, D]          (the block's own keys and values)
 *   LSE              : [B, Hq, S] float32, natural-log log-sum-exp of the
 *                      scaled scores of each row.
 * cache_lens: DEVICE array of B int32 values (4-byte aligned), read by the
 *   kernels only (the host never waits for it).  Values are clamped to
 *   [0, capacity].  capacity <= 2^22; capacity = 0 allows NULL caches.
 * dtype: BD_ATTN_BF16 only (anything else is BD_ATTN_ERR_UNSUPPORTED).
 * The key tiles of all sequences and heads are shared out evenly over a
 * fixed set of waves, whatever the lengths; a KV head's keys split over
 * several waves are merged by a second kernel (the result depends on the
 * lengths of the other sequences only through float32 rounding).
 * ws/ws_bytes: device workspace of at least bd_attn_decode_workspace_bytes
 *   bytes (16-byte aligned; it need not be initialised).
 * Ownership, stream order and errors are as for bd_attn_fwd.
 */
int bd_attn_decode_fwd(const void* Q, const void* K_cache, const void* V_cache, const void* K_new,
                       const void* V_new, const int32_t* cache_lens, int B, int S, int Hq, int Hkv, int D,
                       int capacity, float scale, int dtype, void* O, float* LSE, void* ws, size_t ws_bytes,
                       hipStream_t stream);
/* Workspace bytes for bd_attn_decode_fwd; 0 for arguments it would reject. */
size_t bd_attn_decode_workspace_bytes(int B, int S, int Hq, int Hkv, int D, int capacity, int dtype);

/*
 * Token log-probabilities through the LM head, for the training objectives of
 * blockwise models: the w(t)-weighted cross-entropy over masked positions
 * (Section 2.1, Eq. 3) and the DiPO clipped surrogate with a KL penalty
 * (Section 3.2, Eq. 6-7), both functions of log p(target | position) at the
 * scored positions.  The attention path's output, after the model's last
 * layers, is the input here.
 *
 *   logits[n][v] = sum_d H[n][d] W[v][d]   (never written to memory)
 *   LSE[n]       = log sum_v exp(logits[n][v])
 *   logp[n]      = logits[n][targets[n]] - LSE[n]
 *
 * H: [N, Dm] bf16 (final hidden states of the scored positions), W: [V, Dm]
 * bf16 (LM head), both 16-byte aligned; targets: [N] int32, a target outside
 * [0, V) marks a position that is not scored (logp 0, no gradient).
 * 1 <= N <= 2^22, 1 <= V <= 2^22, Dm a multiple of 256 up to 2^16.  dtype:
 * BD_ATTN_BF16 only.  Float32 accumulation throughout.
 * Ownership, stream order and errors are as for bd_attn_fwd.
 */
int bd_lce_fwd(const void* H, const void* W, const int32_t* targets, int N, int V, int Dm, int dtype,
               float* LSE, float* logp, float* logits, void* ws, size_t ws_bytes, hipStream_t stream);
/*
 * logits (optional, may be NULL): a float32 [N, V rounded up to 256] buffer
 * (bd_lce_logits_bytes, 16-byte aligned) that receives a copy of the logits
 * for bd_lce_bwd, which then skips recomputing them.  Without it the logits
 * exist only tile by tile on chip.
 *
 * Gradients for a per-position coefficient dlogp[n] = dLoss / dlogp[n]
 * (from bd_lce_objective, or any loss of the log-probabilities), given the
 * forward's LSE:
 *   g[n][v] = dlogp[n] (1[v = targets[n]] - exp(logits[n][v] - LSE[n]))
 *   dH = g W  ([N, Dm] bf16),   dW = g^T H  ([V, Dm] bf16).
 * g is formed from the logits kept by bd_lce_fwd when `logits` is not NULL,
 * else recomputed from H and W (one more GEMM), and held in the workspace as
 * bf16 ([N, V rounded up to 256]).
 */
int bd_lce_bwd(const void* H, const void* W, const int32_t* targets, const float* LSE, const float* dlogp,
               const float* logits, int N, int V, int Dm, int dtype, void* dH, void* dW, void* ws, size_t ws_bytes,
               hipStream_t stream);
/* Workspace bytes for bd_lce_fwd (for_bwd = 0) or bd_lce_bwd (for_bwd = 1); 0
 * for arguments they would reject. */
size_t bd_lce_workspace_bytes(int N, int V, int Dm, int dtype, int for_bwd);
/* Bytes of the optional kept-logits buffer; 0 for rejected arguments. */
size_t bd_lce_logits_bytes(int N, int V, int Dm, int dtype);

enum bd_lce_objective_kind { BD_LCE_CE = 0, BD_LCE_DIPO = 1 };
/*
 * Per-position objective values and their derivative dlogp = dloss/dlogp
 * (float32 [N] device arrays; weight carries the per-position factor: the
 * masked-position indicator times w(t) for Eq. 3, or 1 / (total trajectory
 * length) for Eq. 7).
 *   BD_LCE_CE   (Eq. 3):   loss = -weight logp.
 *   BD_LCE_DIPO (Eq. 6-7): r = exp(logp - logp_old),
 *                          s = min(r adv, clip(r, 1 - eps, 1 + eps) adv),
 *                          kl = exp(logp_ref - logp) - (logp_ref - logp) - 1,
 *                          loss = -weight (s - beta kl).
 *     With online updates the behaviour policy is the detached current one:
 *     pass logp itself as logp_old (r = 1).  logp_ref may be NULL when
 *     beta = 0.  eps, beta >= 0.
 */
int bd_lce_objective(const float* logp, const float* logp_old, const float* logp_ref, const float* adv,
                     const float* weight, int N, int kind, float eps, float beta, float* loss, float* dlogp,
                     hipStream_t stream);

/* Comma-separated names of the kernels bd_attn_fwd (for_bwd = 0) or
 * bd_attn_bwd (for_bwd = 1) launch for `dtype`, in launch order (static). */
const char* bd_attn_stage_names(int for_bwd, int dtype);

/* Static, human-readable text for a status code. */
const char* bd_attn_status_string(int status);

/* Library version, major*10000 + minor*100 + patch. */
int bd_attn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* BD_ATTN_H */
