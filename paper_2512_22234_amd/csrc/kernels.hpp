// Kernel argument blocks and launchers shared between the C-ABI layer and the
// kernel translation units.
#pragma once

#include <hip/hip_ext.h>

#include <hip/hip_runtime.h>
#include <stddef.h>

namespace bd {

// Where the sequences lie in the Q-like ([.., Hq, .., D]) and K-like
// ([.., Hkv, .., D]) arrays.
//   Fixed length (cu == nullptr): B sequences of length L; arrays
//     [B][H][2L][D], sequence s's head h at rows (s*H + h)*2L.
//   Packed (cu != nullptr): B sequences with cumulative lengths cu[0..B]
//     (device int32, cu[0] = 0, total T = cu[B]); arrays [H][2T][D],
//     sequence s occupying rows [2 cu[s], 2 cu[s+1]) of every head.  L is
//     then an upper bound on every length (it sizes the grids).
struct SeqLayout {
  const int* cu;
  int T;
  // Length of sequence s, and the first row of its head 0 in the Q-like and
  // the K-like arrays; heads are `hrows` rows apart.
  __device__ void get(int s, int L, int Hq, int Hkv, int& Ls, size_t& qrow, size_t& krow, size_t& hrows) const {
    if (cu == nullptr) {
      Ls = L;
      hrows = 2 * (size_t)L;
      qrow = (size_t)s * Hq * hrows;
      krow = (size_t)s * Hkv * hrows;
    } else {
      // the same for every lane: keep it (and all addresses derived from it) scalar
      const int c0 = __builtin_amdgcn_readfirstlane(cu[s]);
      Ls = __builtin_amdgcn_readfirstlane(cu[s + 1]) - c0;
      hrows = 2 * (size_t)T;
      qrow = krow = 2 * (size_t)c0;
    }
  }
  // The same for a packed sequence whose first token and length are known.
  __device__ void get_packed(int c0, int len, int& Ls, size_t& qrow, size_t& krow, size_t& hrows) const {
    Ls = len;
    hrows = 2 * (size_t)T;
    qrow = krow = 2 * (size_t)c0;
  }
};

// Packed sequences: the tiles of all sequences ranked heaviest first.  Each
// sequence s of length len_s has nt_s = cdiv(len_s, tile) tiles per half;
// row r of the ranking is the pair (s, i) in the order i = ntmax - 1 down to
// 0 and, for one i, the sequences with nt_s > i in order.  (The dK/dV kernel
// ranks its key tiles this way: the work of a key tile grows with the tiles
// after it, so row (s, i) stands for key tile nt_s - 1 - i.)  Every lane of
// the wave calls this with the same r and receives the same result; false
// when r is past the last row.  One ballot per (i, 64 sequences).  Also returns the
// sequence's first token c0 and length len (as SeqLayout::get would read them).
__device__ inline bool packed_row(const int* __restrict__ cu, int n, int ntmax, int tile, int r, int& s_out,
                                  int& i_out, int& nt_out, int& c0_out, int& len_out) {
  const int lane = threadIdx.x & 63;
  int rem = r;
  // up to 64 sequences (one per lane): their bounds are loaded once
  const int lo0 = lane < n ? cu[lane] : 0, hi0 = lane < n ? cu[lane + 1] : 0;
  for (int i = ntmax - 1; i >= 0; --i) {
    for (int base = 0; base < n; base += 64) {
      const int s = base + lane;
      const int lo = base == 0 ? lo0 : s < n ? cu[s] : 0;
      const int hi = base == 0 ? hi0 : s < n ? cu[s + 1] : 0;
      const int nt = (hi - lo + tile - 1) / tile;
      const unsigned long long m = __ballot(nt > i);
      const int cnt = __popcll(m);
      if (rem < cnt) {
        // the rem-th sequence of this chunk with more than i tiles
        const int below = __builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
        const unsigned long long sel = __ballot(nt > i && below == rem);
        const int l = __ffsll((long long)sel) - 1;
        s_out = __builtin_amdgcn_readfirstlane(base + l);
        i_out = i;
        nt_out = __builtin_amdgcn_readfirstlane(__shfl(nt, l));
        c0_out = __builtin_amdgcn_readfirstlane(__shfl(lo, l));
        len_out = __builtin_amdgcn_readfirstlane(__shfl(hi - lo, l));
        return true;
      }
      rem -= cnt;
    }
  }
  return false;
}
// Rows of that ranking: the tiles per half of all sequences.  Same calling
// convention.
__device__ inline int packed_rows(const int* __restrict__ cu, int n, int tile) {
  const int lane = threadIdx.x & 63;
  int sum = 0;
  for (int base = 0; base < n; base += 64) {
    const int s = base + lane;
    sum += s < n ? (cu[s + 1] - cu[s] + tile - 1) / tile : 0;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
  return __builtin_amdgcn_readfirstlane(sum);
}
// Host bound on those rows: sum over s of cdiv(len_s, tile) <= T / tile + n,
// and at most n cdiv(max_L, tile).
inline int packed_rows_bound(int T, int n, int max_L, int tile) {
  const long long a = (long long)T / tile + n, b = (long long)n * ((max_L + tile - 1) / tile);
  return (int)(a < b ? a : b);
}

struct Shape {
  int B, L, S, Hq, Hkv, D;  // B sequences of length L (packed: B sequences, L bounds their lengths)
  int G;                    // Hq / Hkv
  float scale;              // softmax scale (already resolved)
  SeqLayout seq;
};

// Forward tiles: BM queries per workgroup (4 waves x 32), BN keys per step.
constexpr int FWD_BM = 128, FWD_BN = 64;
// dQ tiles: same shape as the forward.
constexpr int DQ_BM = 128, DQ_BN = 64;
// dK/dV tiles: BN keys per workgroup (4 key groups x 32), BM queries per step.
constexpr int DKV_BN = 128, DKV_BM = 32;

// Events a launch records from its own dispatch packet (hipExtLaunchKernelGGL):
// `start` as the kernel begins and `stop` as it ends, with no packet of their
// own in the queue; null events are not recorded.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};

hipError_t launch_cast_f32_to_bf16(const float* x, void* y, size_t n, hipStream_t st, LaunchEvents ev = {});
hipError_t launch_cast_bf16_to_f32(const void* x, float* y, size_t n, hipStream_t st, LaunchEvents ev = {});

hipError_t launch_fwd(const Shape& s, const void* Q, const void* K, const void* V,
                      void* O, float* LSE, hipStream_t st, LaunchEvents ev = {});

// Backward, in launch order:
//   dq:   dQ, and per query row the float32 pair (lse2, delta) =
//         (LSE * log2(e), rowsum(dO * O)) interleaved in rs[2 * row], rs[2 * row + 1]
//         (B*Hq*2L rows); also zeroes the dK/dV pairing counters `pair`.
//   dkdv: dK and dV.  Each clean key tile's walk runs in dkdv_nsplit(s) parts;
//         every part but the last to finish leaves float32 sums in `part`
//         (dkdv_partial_floats elements), the last adds them to its own.
hipError_t launch_bwd_dq(const Shape& s, const void* Q, const void* K, const void* V, const void* dO,
                         const void* O, const float* LSE, float* rs, int* pair, void* dQ, hipStream_t st,
                         LaunchEvents ev = {});
hipError_t launch_bwd_dkdv(const Shape& s, const void* Q, const void* K, const void* V,
                           const void* dO, const float* rs, void* dK, void* dV, float* part, int* pair,
                           hipStream_t st, LaunchEvents ev = {});

// Clean-half key rows of every sequence and KV head: B*Hkv*L for fixed
// length, Hkv*T packed.  Row khead / 2 + k is key k of the clean half of the
// KV head whose position 0 is at K row khead.
inline size_t dkdv_clean_rows(const Shape& s) {
  return s.seq.cu ? (size_t)s.Hkv * s.seq.T : (size_t)s.B * s.Hkv * s.L;
}
// Parts each clean key tile's dK/dV walk is split into: 2, or 4 when half of
// the heaviest walk would be much longer than the average work of one CU, so
// that the kernel would end with its longest items.  Half of key tile 0's
// walk takes about G L / 32 steps; all clean walks of one sequence and KV head
// take about G L (L + 128) / 4096, so over the 256 CUs of the part the ratio is
// 32768 / (nkv (L + 128)), nkv being the sequences times KV heads (for packed
// sequences, the tokens per copy over the longest length).  Results stay
// bitwise reproducible for a given shape: the parts' sums are added in part
// order, whichever finishes first.
constexpr int DKV_CUS = 256;
inline int dkdv_nsplit(int B, int Hkv, int L, const SeqLayout& seq) {
  const double nkv = seq.cu ? (double)Hkv * seq.T / L : (double)B * Hkv;
  const double ratio = (double)DKV_CUS * 128 / (nkv * (L + 128));
  return ratio >= 1.5 ? 4 : 2;
}
inline int dkdv_nsplit(const Shape& s) { return dkdv_nsplit(s.B, s.Hkv, s.L, s.seq); }
// float32 sums of the parts of the clean key tiles' walks that do not finish
// last: per arrival slot (nsplit - 1 of them) and clean key tile (with its
// sequence and KV head: dkdv_tile_slots of them) a region of 2 x 128 x D
// floats (dK and dV of the tile's 128 keys, a ragged last tile padded), in
// the register order of the waves that store and load them.
inline size_t dkdv_tile_slots(const Shape& s) {
  return s.seq.cu ? (size_t)packed_rows_bound(s.seq.T, s.B, s.L, DKV_BN) * s.Hkv
                  : (size_t)((s.L + DKV_BN - 1) / DKV_BN) * s.B * s.Hkv;
}
inline size_t dkdv_partial_floats(const Shape& s) {
  return (size_t)(dkdv_nsplit(s) - 1) * dkdv_tile_slots(s) * 2 * DKV_BN * s.D;
}
// Pairing counters: per (clean key tile, batch x KV head, key group of 32)
// eight ints: the arrival count, the count of parts that have published their
// sums, and for each arrival slot the part index whose sums it holds.
constexpr int DKV_PAIR_INTS = 8;
inline size_t dkdv_pair_ints(int B, int Hkv, int L) {
  return (size_t)DKV_PAIR_INTS * 4 * B * Hkv * ((L + DKV_BN - 1) / DKV_BN);
}

// Block decoding over a KV cache: B sequences, each decoding a block of S
// noisy queries per head against the first cache_lens[b] rows of its cache
// (capacity C) and the block's own S keys.
//   Q, O   : [B][Hq][S][D]      K/V cache : [B][Hkv][C][D]
//   K/V new: [B][Hkv][S][D]     LSE       : [B][Hq][S] float32
// An item is (sequence, KV head, DEC_QT-row tile of the G*S query rows); its
// keys (cache, then block) are cut into DEC_KT-key tiles.  The tiles of all
// items, in item order, are shared out in equal contiguous runs over
// DEC_WAVES waves (DEC_WAVES / 4 workgroups of four).
constexpr int DEC_QT = 32, DEC_KT = 32, DEC_WAVES = 1024;

struct DecodeShape {
  int B, S, Hq, Hkv, D;
  int C;  // cache capacity (rows per sequence and KV head)
  float scale;
};

inline int decode_query_tiles(const DecodeShape& s) { return (s.Hq / s.Hkv * s.S + DEC_QT - 1) / DEC_QT; }
inline size_t decode_items(const DecodeShape& s) { return (size_t)s.B * s.Hkv * decode_query_tiles(s); }
// float32 elements of one partial row: D values, then max and sum (padded to 16 bytes).
inline int decode_part_stride(int D) { return D + 4; }
// Workspace: per item a 16-byte descriptor, then the partial results of every
// (wave, item) run: at most DEC_WAVES + items of them, DEC_QT rows each.
inline size_t decode_desc_bytes(const DecodeShape& s) { return (decode_items(s) * 16 + 255) & ~(size_t)255; }
inline size_t decode_workspace_bytes(const DecodeShape& s) {
  return decode_desc_bytes(s) + (DEC_WAVES + decode_items(s)) * DEC_QT * decode_part_stride(s.D) * 4;
}

// Enqueues the decode kernel and the kernel that merges the runs of items
// shared by several waves.
hipError_t launch_decode(const DecodeShape& s, const void* Q, const void* Kc, const void* Vc, const void* Kn,
                         const void* Vn, const int* cache_lens, void* O, float* LSE, void* ws, hipStream_t st);

// Token log-probabilities through the LM head (H [N][Dm] x W [V][Dm]),
// fused with their softmax.  Dm is a multiple of 256.
constexpr int LCE_BK = 32;  // k per GEMM chunk
struct LceShape {
  int N, V, Dm;
};
inline int lce_vocab_tiles(const LceShape& s) { return (s.V + 255) / 256; }
inline size_t lce_align(size_t x) { return (x + 255) & ~(size_t)255; }
// Forward workspace: per (token, vocabulary tile) the partial (max, sum).
inline size_t lce_fwd_part_offset(const LceShape&) { return 0; }
inline size_t lce_fwd_workspace_bytes(const LceShape& s) { return lce_align((size_t)s.N * lce_vocab_tiles(s) * 8); }
// Backward workspace: g = coef (onehot - softmax) as bf16 [N][V rounded up to 256].
inline size_t lce_bwd_g_offset(const LceShape&) { return 0; }
inline size_t lce_bwd_workspace_bytes(const LceShape& s) {
  return lce_align((size_t)s.N * lce_vocab_tiles(s) * 256 * 2);
}

// Kept logits (optional): float32 [N][V rounded up to 256].
inline size_t lce_logits_bytes(const LceShape& s) { return (size_t)s.N * lce_vocab_tiles(s) * 256 * 4; }
hipError_t launch_lce_fwd(const LceShape& s, const void* H, const void* W, const int* targets, float* lse,
                          float* logp, float* logits, void* ws, hipStream_t st);
hipError_t launch_lce_bwd(const LceShape& s, const void* H, const void* W, const int* targets, const float* lse,
                          const float* coef, const float* logits, void* dH, void* dW, void* ws, hipStream_t st);
hipError_t launch_lce_objective(int N, int kind, float eps, float beta, const float* logp, const float* logp_old,
                                const float* logp_ref, const float* adv, const float* weight, float* loss,
                                float* dlogp, hipStream_t st);

}  // namespace bd
