// Token log-probabilities through the LM head, fused with their softmax, for
// the blockwise objectives of DiRL: the w(t)-weighted cross-entropy over
// masked positions (Section 2.1, Eq. 3) and the DiPO / GRPO clipped
// surrogate with a KL penalty (Section 3.2, Eq. 6-7), both functions of
// log p(target | position) at the scored positions.
//
//   logits[n][v] = sum_d H[n][d] W[v][d]            (H: [N][Dm], W: [V][Dm], bf16)
//   LSE[n]       = log sum_v exp(logits[n][v])
//   logp[n]      = logits[n][t_n] - LSE[n]
// and, for a per-token coefficient c_n = dLoss / dlogp_n,
//   g[n][v] = c_n (1[v = t_n] - exp(logits[n][v] - LSE[n]))
//   dH = g W,   dW = g^T H.
//
// The target logit of each token is one float32 dot product (merge and
// one-hot kernels), so the tile epilogues carry no per-element target test.
// The logits never reach HBM.  Every product is one GEMM kernel: 256 x 256
// output tiles, four waves of 128 x 128, k in chunks of 32 through a
// four-stage LDS ring (HBM/L2 -> LDS copies three chunks ahead), one
// workgroup barrier per chunk placed mid-chunk so that the operand reads of
// the next chunk overlap the MFMAs of the current one.  An operand tile is
// either ROW (256 rows of 32 k values: the k index is contiguous in memory)
// or TR (32 k rows of 256 values: the other index is contiguous), read with
// row-slice or transposing LDS reads in the same k order.  Output rows are
// the B side of the MFMA, so each lane holds four consecutive output columns
// and the epilogues stage whole 512-byte rows through LDS.
//
//   kernel  A side (MFMA A, output columns)  B side (MFMA B, output rows)  K    epilogue
//   FWD     W, ROW (vocab)                   H, ROW (tokens)               Dm   (max, sum) per token and vocab tile
//   REC     W, ROW                           H, ROW                        Dm   g -> G [N][Vp] bf16 (target entry afterwards)
// (the forward can also keep its float32 logits, [N][Vp]; the backward then
// forms g from them elementwise instead of running REC)
//   DH      W, TR  (k = vocab, cols = d)     G, ROW (tokens)               Vp   dH [N][Dm]
//   DW      H, TR  (k = tokens, cols = d)    G, TR  (k = tokens, vocab)    N    dW [V][Dm]
#include "device.hpp"
#include "kernels.hpp"

namespace bd {
namespace {

constexpr int TB = 256;               // output tile (both sides)
constexpr int BK = LCE_BK;            // k per chunk
constexpr int NST = 4;                // LDS ring stages
constexpr uint32_t OPB = TB * BK * 2;  // bytes of one operand tile (16 KB)
constexpr int RED_STRIDE = TB + 8;    // staging row stride (bf16) of the output tile: 528 bytes

// EPI_FWD_KEEP is EPI_FWD that also stores the float32 logits (a variant of
// its own, so the plain forward's epilogue carries none of its registers)
enum Epi { EPI_FWD = 0, EPI_REC = 1, EPI_STORE = 2, EPI_FWD_KEEP = 3 };

struct LceParams {
  const bf16* A;  // A-side source
  const bf16* B;  // B-side source
  int lda, ldb;   // row strides (elements)
  int a_ext, b_ext;  // ROW: valid rows of the side; TR: valid k rows
  int Mcols, Nrows;  // output columns (A side) and rows (B side) that exist
  int K;             // k extent rounded up to BK (padding reads as zero)
  int nMT, nNT;      // tiles along the A and B sides
  // epilogue
  const int* targets;  // [N]
  const float* coef;   // [N]
  const float* lse;    // [N]
  float* part;         // FWD: [N][nMT] (max in log2 units, sum)
  float* logits;       // FWD: optional [N][ldl] float32 copy of the logits (null: not kept)
  int ldl;
  bf16* C;             // REC: G [N][ldc]; STORE: dH or dW
  int ldc;
  int V;               // vocabulary size (FWD/REC: valid A-side columns)
};

// Tile order: super-blocks of 4 (A side) x 8 (B side) tiles, dealt to the 8
// XCDs in turn (workgroups are dispatched round-robin over the XCDs), so the
// 32 workgroups an XCD runs at once share 4 A tiles and 8 B tiles in its L2.
constexpr int GM = 4, GN = 8;

// Buffer resource built from values that are the same in every lane: taking
// them through readfirstlane keeps the descriptor in scalar registers (a
// descriptor the compiler cannot prove uniform costs a loop per copy).
__device__ inline __amdgpu_buffer_rsrc_t uniform_buffer(const void* base, size_t bytes) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a), hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  const uint32_t n = __builtin_amdgcn_readfirstlane((uint32_t)bytes);
  return make_buffer((const void*)(uintptr_t)(((uint64_t)hi << 32) | lo), n);
}

template <bool TR>
struct OperandCopy;

// ROW: 256 rows x 32 k (64-byte rows, swizzled); a wave copies 4 KB per chunk.
template <>
struct OperandCopy<false> {
  uint32_t off[4];  // byte offset of this lane's 16 bytes for instruction u, within rows of stride ld
  __device__ OperandCopy(int w, int lane, int ld) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int p = (u * 4 + w) * 64 + lane;  // 16-byte chunk of the LDS tile
      const int r = p >> 2, c = (p & 3) ^ chunk_swizzle<BK>(r);
      off[u] = (uint32_t)(2 * ((size_t)r * ld + c * 8));
    }
  }
  // rows [r0, r0 + 256) of src (valid below ext), k columns [k0, k0 + 32); w: this wave (uniform)
  __device__ void issue(const bf16* src, int ld, int ext, int r0, int k0, char* dst, int w) const {
    const int rows = imin(TB, ext - r0);
    const __amdgpu_buffer_rsrc_t rs = uniform_buffer(src + (size_t)r0 * ld, (size_t)imax(rows, 0) * ld * 2);
#pragma unroll
    for (int u = 0; u < 4; ++u)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(dst + (u * 4 + w) * 1024),
                                               16, (int)(off[u] + 2 * k0), 0, 0, 0);
  }
};

// TR: 32 k rows x 256 columns, as two 32 x 128 sub-tiles (256-byte rows).
template <>
struct OperandCopy<true> {
  uint32_t off[4];
  __device__ OperandCopy(int w, int lane, int ld) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int sub = u >> 1;
      const int p = ((u & 1) * 4 + w) * 64 + lane;  // 16-byte chunk of the sub-tile
      const int r = p >> 4, c = (p & 15) ^ chunk_swizzle<128>(r);
      off[u] = (uint32_t)(2 * ((size_t)r * ld + sub * 128 + c * 8));
    }
  }
  // k rows [k0, k0 + 32) of src (valid below ext), columns [c0, c0 + 256); w: this wave (uniform)
  __device__ void issue(const bf16* src, int ld, int ext, int c0, int k0, char* dst, int w) const {
    const int rows = imin(BK, ext - k0);
    const __amdgpu_buffer_rsrc_t rs = uniform_buffer(src + (size_t)k0 * ld + c0, (size_t)imax(rows, 0) * ld * 2);
#pragma unroll
    for (int u = 0; u < 4; ++u)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rs, (__attribute__((address_space(3))) void*)(dst + (u >> 1) * (OPB / 2) + ((u & 1) * 4 + w) * 1024), 16,
          (int)off[u], 0, 0, 0);
  }
};

// MFMA operand of 32-block `blk` (0..7) of a side, k16 step s (0, 1) of the chunk.
struct OperandRead {
  uint32_t row_rel;     // ROW tiles
  uint32_t tr0, tr1;    // TR tiles (linear k order)
  __device__ explicit OperandRead(int lane) {
    const LdsOperands<BK> o(lane);
    row_rel = o.row_rel;
    const LdsLinearTr<128> t(lane);
    tr0 = t.rel0;
    tr1 = t.rel1;
  }
  template <bool TR>
  __device__ bf16x8 get(const char* tile, int s, int blk) const {
    if constexpr (TR) return lds_tr<128>(tile + (blk >> 2) * (OPB / 2), tr0, tr1, s, blk & 3);
    else return lds_rows<BK>(tile, row_rel, s, blk);
  }
};

struct LceSmem {
  alignas(256) char a[NST][OPB];
  alignas(256) char b[NST][OPB];
  float2 red[2][TB];  // FWD: per token row, the two A-half waves' (max, sum)
};
// The output tile is staged over the ring once the k loop is done.
static_assert(sizeof(LceSmem) >= TB * RED_STRIDE * 2, "staging fits in the ring");

template <int EPI, bool ATR, bool BTR>
__global__ __launch_bounds__(256, 1) void lce_gemm_kernel(LceParams p) {
  __shared__ LceSmem sm;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, g2 = lane >> 5;
  const int wa = w & 1, wb = w >> 1;  // this wave's 128-wide halves of the A and B sides

  // tile of this workgroup
  const int id = blockIdx.x, xcd = id & 7, slot = id >> 3;
  const int nBN = cdiv(p.nNT, GN);
  const int blk = (slot / (GM * GN)) * 8 + xcd, within = slot % (GM * GN);
  const int mt = (blk / nBN) * GM + within % GM, nt = (blk % nBN) * GN + within / GM;
  if (mt >= p.nMT || nt >= p.nNT) return;
  const int m0 = mt * TB, n0 = nt * TB;

  const OperandCopy<ATR> ca(w, lane, p.lda);
  const OperandCopy<BTR> cb(w, lane, p.ldb);
  const OperandRead rd(lane);
  auto issue = [&](int kc, char* da, char* db) {
    const int k0 = kc * BK;
    ca.issue(p.A, p.lda, p.a_ext, m0, k0, da, w);
    cb.issue(p.B, p.ldb, p.b_ext, n0, k0, db, w);
  };
  const int nk = p.K / BK;
  constexpr int NI = 8;  // copy instructions per wave per chunk

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

#pragma unroll
  for (int c = 0; c < NST - 1; ++c) issue(imin(c, nk - 1), sm.a[c], sm.b[c]);
  wait_global_loads_but<(NST - 2) * NI>();  // chunk 0 has landed
  __syncthreads();

  bf16x8 a0[4], b0[4], a1[4], b1[4];
  auto read = [&](const char* ta, const char* tb, int s, bf16x8* a, bf16x8* b) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = rd.get<ATR>(ta, s, 4 * wa + i);
#pragma unroll
    for (int j = 0; j < 4; ++j) b[j] = rd.get<BTR>(tb, s, 4 * wb + j);
  };
  auto mm = [&](const bf16x8* a, const bf16x8* b) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = mfma32(a[i], b[j], acc[i][j]);
  };
  // LDS reads per k16 step: 8 for ROW/ROW, up to 16 for TR/TR (a transposing
  // operand takes two 8-byte reads)
  constexpr int RPS = (ATR ? 8 : 4) + (BTR ? 8 : 4);
  // Chunk kc, step 0's operands already in (a0, b0):
  //   step 0 MFMAs beside the reads of step 1;
  //   wait for chunk kc + 1, barrier (all copies in; all waves done with chunk kc - 1);
  //   copy chunk kc + 3 into chunk kc - 1's stage;
  //   step 1 MFMAs beside the reads of chunk kc + 1's step 0.
  auto half1 = [&](const char* __restrict__ ta, const char* __restrict__ tb) __attribute__((always_inline)) {
    read(ta, tb, 1, a1, b1);
    mm(a0, b0);
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (q < RPS) __builtin_amdgcn_sched_group_barrier(0x100, RPS > 16 ? 2 : 1, 0);
    }
  };
  auto half2 = [&](const char* __restrict__ ta, const char* __restrict__ tb, char* __restrict__ wa_, char* __restrict__ wb_,
                   int kc) __attribute__((always_inline)) {
    issue(imin(kc + NST - 1, nk - 1), wa_, wb_);
    read(ta, tb, 0, a0, b0);
    mm(a1, b1);
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (q < RPS) __builtin_amdgcn_sched_group_barrier(0x100, RPS > 16 ? 2 : 1, 0);
      if (q < NI) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    }
  };
  read(sm.a[0], sm.b[0], 0, a0, b0);
  for (int kc = 0; kc < nk; ++kc) {
    const int st = kc % NST, s1 = (kc + 1) % NST, sw = (kc + NST - 1) % NST;
    half1(sm.a[st], sm.b[st]);
    compute_fence();
    wait_global_loads_but<(NST - 3) * NI>();  // chunk kc + 1 has landed (this wave's part)
    barrier_lds_only();
    half2(sm.a[s1], sm.b[s1], sm.a[sw], sm.b[sw], kc);
    compute_fence();
  }
  wait_global_loads();  // the last (repeated) copies, before the ring is reused
  __syncthreads();

  // acc[i][j][4 i4 + jj]: A-side column  m0 + 128 wa + 32 i + 8 i4 + 4 g2 + jj,
  //                       B-side row     n0 + 128 wb + 32 j + l32
  // Columns past the vocabulary exist only in the last vocabulary tile.
  const bool partial_cols = m0 + TB > p.V;
  if constexpr (EPI == EPI_FWD || EPI == EPI_FWD_KEEP) {
    // per token: max and sum of exp over this tile's vocabulary columns (log2
    // units).  Every tile takes the masked path: a branch between a masked and
    // an unmasked copy makes the compiler move all 256 accumulators into VGPRs
    // ahead of it, which spills.
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      // scores recomputed from the accumulators in each pass (nothing is
      // written back, so no block's values stay live longer)
      auto score = [&](int i, int e) __attribute__((always_inline)) {
        const int v = m0 + 128 * wa + 32 * i + 8 * (e >> 2) + 4 * g2 + (e & 3);
        return v < p.V ? acc[i][j][e] * LOG2E : -INFINITY;
      };
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) mx = fmaxf(mx, score(i, e));
      mx = halves_max(mx);
      float sum = 0.f;
      if (mx != -INFINITY) {  // (a wave half past the last vocabulary row has no columns)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int e = 0; e < 16; ++e) sum += fast_exp2(score(i, e) - mx);  // exp2(-inf) = 0
      }
      sum = halves_sum(sum);
      if (g2 == 0) sm.red[wa][128 * wb + 32 * j + l32] = float2{mx, sum};
    }
    if constexpr (EPI == EPI_FWD_KEEP) {
      // the logits for the backward pass (columns past V hold the zero rows'
      // logits, 0)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int n = n0 + 128 * wb + 32 * j + l32;
        if (n < p.Nrows) {
          float* lr = p.logits + (size_t)n * p.ldl + m0 + 128 * wa + 4 * g2;
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int i4 = 0; i4 < 4; ++i4)
              *reinterpret_cast<f32x4*>(lr + 32 * i + 8 * i4) =
                  f32x4{acc[i][j][4 * i4], acc[i][j][4 * i4 + 1], acc[i][j][4 * i4 + 2], acc[i][j][4 * i4 + 3]};
        }
      }
    }
    barrier_lds_only();  // (the kept-logits stores need not have landed: only LDS is exchanged)
    // two halves of the vocabulary tile -> one partial per token
    const int n = n0 + tid;
    if (n < p.Nrows) {
      const float2 x = sm.red[0][tid], y = sm.red[1][tid];
      const float M = fmaxf(x.x, y.x);  // finite: every tile holds at least one vocabulary row
      const float S = x.y * fast_exp2(x.x - M) + y.y * fast_exp2(y.x - M);
      *reinterpret_cast<float2*>(p.part + 2 * ((size_t)n * p.nMT + mt)) = float2{M, S};
    }
  } else {
    // stage the bf16 output tile, rows = B side, 4 consecutive columns per lane and (i, i4)
    bf16* stg = reinterpret_cast<bf16*>(&sm);
    auto stage = [&](auto masked) __attribute__((always_inline)) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int rloc = 128 * wb + 32 * j + l32, n = n0 + rloc;
        // REC: g = -c p off the target column (the target entry is rewritten afterwards)
        float ncf = 0.f, l2 = 0.f;
        if constexpr (EPI == EPI_REC) {
          if (n < p.Nrows) {
            const int t = p.targets[n];
            ncf = (t >= 0 && t < p.V) ? -p.coef[n] : 0.f;
            l2 = p.lse[n] * LOG2E;
          }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int i4 = 0; i4 < 4; ++i4) {
            const int cloc = 128 * wa + 32 * i + 8 * i4 + 4 * g2;
            float o[4];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
              float x = acc[i][j][4 * i4 + jj];
              if constexpr (EPI == EPI_REC) {
                x = ncf * fast_exp2(x * LOG2E - l2);
                if constexpr (decltype(masked)::value) x = m0 + cloc + jj < p.V ? x : 0.f;
              }
              o[jj] = x;
            }
            st_bf16x4(stg + rloc * RED_STRIDE + cloc, o[0], o[1], o[2], o[3]);
          }
      }
    };
    if (EPI == EPI_REC && partial_cols) stage(Flag<true>());
    else stage(Flag<false>());
    barrier_lds_only();  // the staged tile is in LDS
    // write rows of 256 columns (512 bytes): 16 lanes a row, 16 bytes each
    const int cr = (tid & 15) * 16;
#pragma unroll 4
    for (int r = tid >> 4; r < TB; r += 16) {
      const int n = n0 + r;
      if (n >= p.Nrows) break;
      const int c = m0 + cr;
      if (c >= p.Mcols) continue;
      const u32x4 v0 = *reinterpret_cast<const u32x4*>(stg + r * RED_STRIDE + cr);
      const u32x4 v1 = *reinterpret_cast<const u32x4*>(stg + r * RED_STRIDE + cr + 8);
      bf16* dst = p.C + (size_t)n * p.ldc + c;
      *reinterpret_cast<u32x4*>(dst) = v0;
      *reinterpret_cast<u32x4*>(dst + 8) = v1;
    }
  }
}

// logits[n][t] = H[n] . W[t] in float32, by one wave (16-byte loads).
__device__ inline float lce_target_logit(const bf16* H, const bf16* W, int Dm, int n, int t, int lane) {
  const bf16* h = H + (size_t)n * Dm;
  const bf16* wr = W + (size_t)t * Dm;
  float acc = 0.f;
  for (int d = 8 * lane; d < Dm; d += 512) {
    const bf16x8 x = *reinterpret_cast<const bf16x8*>(h + d);
    const bf16x8 y = *reinterpret_cast<const bf16x8*>(wr + d);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc += (float)x[e] * (float)y[e];
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
  return acc;
}

// Per token: LSE from the per-tile partials and logp of the target.  One wave
// per token.
__global__ __launch_bounds__(256) void lce_merge_kernel(const float* part, const bf16* H, const bf16* W,
                                                       const int* targets, int N, int nMT, int V, int Dm, float* lse,
                                                       float* logp) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  const float2* pp = reinterpret_cast<const float2*>(part) + (size_t)n * nMT;
  float M = -INFINITY;
  for (int t = lane; t < nMT; t += 64) M = fmaxf(M, pp[t].x);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) M = fmaxf(M, __shfl_xor(M, o, 64));
  float S = 0.f;
  for (int t = lane; t < nMT; t += 64) {
    const float2 x = pp[t];
    S += x.y * fast_exp2(x.x - M);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) S += __shfl_xor(S, o, 64);
  const int t = targets[n];
  const bool valid = t >= 0 && t < V;
  const float tl = valid ? lce_target_logit(H, W, Dm, n, t, lane) : 0.f;
  if (lane == 0) {
    const float l = (M + __log2f(S)) * LN2;
    lse[n] = l;
    logp[n] = valid ? tl - l : 0.f;
  }
}

// g = -c exp(logit - LSE) from kept logits, bf16, zero past V (the target
// entries are rewritten by lce_onehot_kernel).  One thread per 8 columns.
__global__ __launch_bounds__(256) void lce_g_from_logits_kernel(const float* logits, const int* targets,
                                                               const float* lse, const float* coef, int N, int V,
                                                               int Vp, bf16* G) {
  const size_t id = (size_t)blockIdx.x * 256 + threadIdx.x;
  const int per = Vp / 8;
  const size_t n = id / per;
  if (n >= (size_t)N) return;
  const int v0 = (int)(id % per) * 8;
  const int t = targets[n];
  const float ncf = (t >= 0 && t < V) ? -coef[n] : 0.f;
  const float l2 = lse[n] * LOG2E;
  const float* x = logits + n * Vp + v0;
  const f32x4 a = *reinterpret_cast<const f32x4*>(x), b = *reinterpret_cast<const f32x4*>(x + 4);
  bf16x8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float xe = e < 4 ? a[e] : b[e - 4];
    o[e] = (bf16)(v0 + e < V ? ncf * fast_exp2(xe * LOG2E - l2) : 0.f);
  }
  *reinterpret_cast<bf16x8*>(G + n * Vp + v0) = o;
}

// The target entry of g: c (1 - p_t), from the target logit in float32 (the
// tile epilogue wrote -c p_t there).  One wave per token.
__global__ __launch_bounds__(256) void lce_onehot_kernel(const bf16* H, const bf16* W, const int* targets,
                                                        const float* lse, const float* coef, int N, int V, int Dm,
                                                        bf16* G, int ldg) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  const int t = targets[n];
  if (t < 0 || t >= V) return;
  const float tl = lce_target_logit(H, W, Dm, n, t, lane);
  if (lane == 0) G[(size_t)n * ldg + t] = (bf16)(coef[n] * (1.f - __expf(tl - lse[n])));
}

// Per-token objectives and their derivative with respect to logp.
//   kind 0 (Eq. 3):   loss = -w logp                         dloss/dlogp = -w
//   kind 1 (Eq. 6-7): r = exp(logp - logp_old),
//                     s = min(r A, clip(r, 1 - eps, 1 + eps) A),
//                     kl = exp(logp_ref - logp) - (logp_ref - logp) - 1,
//                     loss = -w (s - beta kl)
//                     dloss/dlogp = -w (ds/dlogp - beta dkl/dlogp),
//                     ds/dlogp = r A where the unclipped term is the minimum, else 0,
//                     dkl/dlogp = 1 - exp(logp_ref - logp).
__global__ __launch_bounds__(256) void lce_objective_kernel(const float* logp, const float* logp_old,
                                                           const float* logp_ref, const float* adv,
                                                           const float* weight, int N, int kind, float eps,
                                                           float beta, float* loss, float* dlogp) {
  const int n = blockIdx.x * 256 + threadIdx.x;
  if (n >= N) return;
  const float lp = logp[n], w = weight[n];
  if (kind == 0) {
    loss[n] = -w * lp;
    dlogp[n] = -w;
    return;
  }
  const float a = adv[n];
  const float r = __expf(lp - logp_old[n]);
  const float rc = fminf(fmaxf(r, 1.f - eps), 1.f + eps);
  const float un = r * a, cl = rc * a;
  const bool use_un = un <= cl;  // the minimum; at a tie both terms agree and r is inside the clip range
  const float s = use_un ? un : cl;
  const float ds = use_un ? un : 0.f;
  float kl = 0.f, dkl = 0.f;
  if (beta != 0.f) {
    const float d = logp_ref[n] - lp, ed = __expf(d);
    kl = ed - d - 1.f;
    dkl = 1.f - ed;
  }
  loss[n] = -w * (s - beta * kl);
  dlogp[n] = -w * (ds - beta * dkl);
}

template <int EPI, bool ATR, bool BTR>
hipError_t launch_gemm(const LceParams& p, hipStream_t st) {
  const int nBM = cdiv(p.nMT, GM), nBN = cdiv(p.nNT, GN);
  const int grid = cdiv(nBM * nBN, 8) * 8 * GM * GN;
  hipLaunchKernelGGL((lce_gemm_kernel<EPI, ATR, BTR>), dim3(grid), dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_lce_fwd(const LceShape& s, const void* H, const void* W, const int* targets, float* lse,
                          float* logp, float* logits, void* ws, hipStream_t st) {
  LceParams p{};
  p.A = static_cast<const bf16*>(W);
  p.B = static_cast<const bf16*>(H);
  p.lda = p.ldb = s.Dm;
  p.a_ext = s.V;
  p.b_ext = s.N;
  p.Mcols = s.V;
  p.Nrows = s.N;
  p.K = s.Dm;
  p.nMT = lce_vocab_tiles(s);
  p.nNT = cdiv(s.N, TB);
  p.targets = targets;
  char* w = static_cast<char*>(ws);
  p.part = reinterpret_cast<float*>(w + lce_fwd_part_offset(s));
  p.logits = logits;
  p.ldl = lce_vocab_tiles(s) * TB;
  p.V = s.V;
  hipError_t e = logits != nullptr ? launch_gemm<EPI_FWD_KEEP, false, false>(p, st)
                                    : launch_gemm<EPI_FWD, false, false>(p, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(lce_merge_kernel, dim3(cdiv(s.N, 4)), dim3(256), 0, st, p.part, p.B, p.A, targets, s.N, p.nMT,
                     s.V, s.Dm, lse, logp);
  return hipGetLastError();
}

hipError_t launch_lce_objective(int N, int kind, float eps, float beta, const float* logp, const float* logp_old,
                                const float* logp_ref, const float* adv, const float* weight, float* loss,
                                float* dlogp, hipStream_t st) {
  hipLaunchKernelGGL(lce_objective_kernel, dim3(cdiv(N, 256)), dim3(256), 0, st, logp, logp_old, logp_ref, adv,
                     weight, N, kind, eps, beta, loss, dlogp);
  return hipGetLastError();
}

hipError_t launch_lce_bwd(const LceShape& s, const void* H, const void* W, const int* targets, const float* lse,
                          const float* coef, const float* logits, void* dH, void* dW, void* ws, hipStream_t st) {
  const int Vp = lce_vocab_tiles(s) * TB;
  bf16* G = reinterpret_cast<bf16*>(static_cast<char*>(ws) + lce_bwd_g_offset(s));
  // G = coef (onehot - softmax), [N][Vp] (columns past V zero)
  LceParams p{};
  p.A = static_cast<const bf16*>(W);
  p.B = static_cast<const bf16*>(H);
  p.lda = p.ldb = s.Dm;
  p.a_ext = s.V;
  p.b_ext = s.N;
  p.Mcols = Vp;
  p.Nrows = s.N;
  p.K = s.Dm;
  p.nMT = lce_vocab_tiles(s);
  p.nNT = cdiv(s.N, TB);
  p.targets = targets;
  p.coef = coef;
  p.lse = lse;
  p.C = G;
  p.ldc = Vp;
  p.V = s.V;
  hipError_t e;
  if (logits != nullptr) {
    const size_t threads = (size_t)s.N * (Vp / 8);
    hipLaunchKernelGGL(lce_g_from_logits_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st, logits,
                       targets, lse, coef, s.N, s.V, Vp, G);
    e = hipGetLastError();
  } else {
    e = launch_gemm<EPI_REC, false, false>(p, st);
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(lce_onehot_kernel, dim3(cdiv(s.N, 4)), dim3(256), 0, st, p.B, p.A, targets, lse, coef, s.N,
                     s.V, s.Dm, G, Vp);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // dH[n][d] = sum_v G[n][v] W[v][d]
  LceParams q{};
  q.A = static_cast<const bf16*>(W);
  q.B = G;
  q.lda = s.Dm;
  q.ldb = Vp;
  q.a_ext = s.V;
  q.b_ext = s.N;
  q.Mcols = s.Dm;
  q.Nrows = s.N;
  q.K = Vp;
  q.nMT = s.Dm / TB;
  q.nNT = cdiv(s.N, TB);
  q.C = static_cast<bf16*>(dH);
  q.ldc = s.Dm;
  e = launch_gemm<EPI_STORE, true, false>(q, st);
  if (e != hipSuccess) return e;
  // dW[v][d] = sum_n G[n][v] H[n][d]
  LceParams r{};
  r.A = static_cast<const bf16*>(H);
  r.B = G;
  r.lda = s.Dm;
  r.ldb = Vp;
  r.a_ext = s.N;
  r.b_ext = s.N;
  r.Mcols = s.Dm;
  r.Nrows = s.V;
  r.K = cdiv(s.N, BK) * BK;
  r.nMT = s.Dm / TB;
  r.nNT = lce_vocab_tiles(s);
  r.C = static_cast<bf16*>(dW);
  r.ldc = s.Dm;
  return launch_gemm<EPI_STORE, true, true>(r, st);
}

}  // namespace bd
