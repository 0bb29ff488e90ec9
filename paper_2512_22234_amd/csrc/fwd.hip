// Forward pass of block-diffusion masked attention (DiRL Section 4.1, mask of
// Eq. 1 / Eq. 2) for gfx950.
//
// One workgroup = one (batch, query head, query tile of 128 rows); four waves,
// each owning 32 query rows.  Scores are computed transposed, S^T = K Q^T, so
// that each lane owns one query column: the row max needs one cross-lane
// exchange (lane l <-> l+32) per key tile and the running row sum stays a
// per-lane partial until the epilogue.  O^T = V^T P^T reuses the score
// accumulator directly as the bf16 B operand; its A operand V^T is read from
// the V tile with the transposing LDS read (see device.hpp).
//
// Key tiles (64 keys) are visited in the order given by the exact tile
// classification: FULL tiles run with no per-element test, PARTIAL tiles
// apply the visibility window per element, EMPTY tiles are never loaded.  K
// and V tiles are copied into LDS asynchronously (buffer loads to LDS) one
// tile ahead, double-buffered, so the copy runs under the current tile's
// compute.
// The online softmax keeps a reference maximum per row that only moves when
// the scores exceed it by a margin, so the O rescale is rare.
#include "device.hpp"
#include "kernels.hpp"

namespace bd {
namespace {

struct FwdParams {
  const bf16* Q;
  const bf16* K;
  const bf16* V;
  bf16* O;
  float* LSE;
  SeqLayout seq;
  int L, S, Hq, Hkv, G, nQT, nbh;  // L: the (maximum) sequence length; nbh: sequences x query heads
  float c;  // scale * log2(e)
};

template <int D>
struct FwdSmem {
  static constexpr int BN = FWD_BN;
  static constexpr uint32_t TILE = BN * D * 2;  // bytes per swizzled tile
  bf16 k[2][BN * D];  // byte offset buf * TILE
  bf16 v[2][BN * D];  // byte offset (2 + buf) * TILE
};

// The reference maximum of a row moves only when the row's scores exceed it
// by more than this (log2 units), so the accumulator rescale is rare; P stays
// below 2^8 and the final O / l and LSE are unchanged (both use the same
// reference).
constexpr float RESCALE_SLACK = 8.0f;

// Maximum of N values as a balanced tree (depth log2 N instead of a chain of N).
template <int N>
__device__ inline float tree_max(const float* v) {
  if constexpr (N == 1) {
    return v[0];
  } else {
    return fmaxf(tree_max<N / 2>(v), tree_max<N - N / 2>(v + N / 2));
  }
}
// Sum of the 16 K entries of K accumulators as a balanced tree.
template <int K>
__device__ inline float tree_sum(const f32x16* a) {
  float t[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    t[e] = a[0][e];
#pragma unroll
    for (int k = 1; k < K; ++k) t[e] += a[k][e];
  }
#pragma unroll
  for (int w = 8; w > 0; w >>= 1)
#pragma unroll
    for (int e = 0; e < w; ++e) t[e] += t[e + w];
  return t[0];
}

template <int D>
__global__ __launch_bounds__(256, 2) void fwd_kernel(FwdParams p) {
  constexpr int BM = FWD_BM, BN = FWD_BN;
  constexpr int DS = D / 16, DB = D / 32, KB = BN / 32, PC = BN / 16;
  constexpr uint32_t TILE = FwdSmem<D>::TILE;
  __shared__ FwdSmem<D> sm;
  char* lds = reinterpret_cast<char*>(&sm);

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, g2 = lane >> 5;

  // Heaviest query tiles first (work grows with the tile index), noisy before
  // clean; heads remapped so a KV group stays on one XCD.
  const int id = blockIdx.x;
  const int rank = id / p.nbh;
  const int bh = xcd_head_remap(id - rank * p.nbh, p.nbh, p.G);
  const int qi = p.nQT - 1 - (rank >> 1);
  const int qh = rank & 1;
  const int b = bh / p.Hq, hq = bh - b * p.Hq, hk = hq / p.G;
  // sequence b: its length and where its rows lie
  int L;
  size_t qrow0, krow0, hrows;
  p.seq.get(b, p.L, p.Hq, p.Hkv, L, qrow0, krow0, hrows);
  if (qi * BM >= L) return;  // a shorter sequence than the grid is sized for (whole workgroup)
  // (a sequence shorter than S is one block: every formula below gives
  // the S = L mask then)
  const int S = p.S;
  const int N = 2 * L;
  const int q0 = qi * BM, q1 = imin(L, q0 + BM);

  const size_t kvbase = (krow0 + hk * hrows) * D;
  const size_t qbase = qrow0 + hq * hrows;  // row of this head's position 0 in Q, O and LSE

  const int r = q0 + w * 32 + l32;  // this lane's query row (local to its half)
  const bool qvalid = r < q1;
  const int qblock0 = qvalid ? (r / S) * S : 0;
  const int prow = qh * L + r;

  const KeyTileList kl = key_tiles_for_query_tile(qh, qi, L, S, BM, BN);
  const int T = __builtin_amdgcn_readfirstlane(kl.count());  // (uniform; keeps the step loops scalar)
  const TileCopy<D, BN, 256> copy(tid);
  const bf16* const kbase = p.K + kvbase;
  const bf16* const vbase = p.V + kvbase;
  // first packed row of key tile t (2L rows for this batch and KV head)
  auto tile_row = [&](int t) {
    int kh, j;
    kl.at(t, kh, j);
    return kh * L + j * BN;
  };
  // copy key tile t of K or V
  auto issue = [&](int t, bool is_v, char* dst) {
    // (the row is the same for every lane; saying so keeps the copy's buffer
    // descriptor scalar where the compiler cannot prove it)
    const int r = __builtin_amdgcn_readfirstlane(tile_row(t));
    copy.issue_rows((is_v ? vbase : kbase) + (size_t)r * D, N - r, dst);
  };

  if (T > 0) {
    issue(0, false, lds);
    issue(0, true, lds + 2 * TILE);
  }

  bf16x8 qreg[DS];
  {
    const bf16* qp = p.Q + (qbase + prow) * D + 8 * g2;
#pragma unroll
    for (int s = 0; s < DS; ++s)
      qreg[s] = qvalid ? *reinterpret_cast<const bf16x8*>(qp + 16 * s) : zero_bf16x8();
  }
  const LdsOperands<D> ops(lane);

  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[db][e] = 0.f;
  float m = -INFINITY, lsum = 0.f;  // reference max (log2 units) and row sum relative to it

  wait_global_loads();
  __syncthreads();

  // Per-step bookkeeping is a few scalar instructions: the FULL test is two
  // comparisons against per-workgroup bounds and the visibility windows of
  // both key halves are computed once.
  const FullRange fr = full_range_vs_query_tile(qh, q0, q1, L, S, BM);
  const PosWindow win_n = keys_visible_from(qh, HALF_NOISY, qblock0, L, S, qvalid);
  const PosWindow win_c = keys_visible_from(qh, HALF_CLEAN, qblock0, L, S, qvalid);
  // The keys any row of this wave can see, per half (a wave-uniform union of
  // the rows' windows): on the diagonal tiles a 32-key block outside it is
  // skipped by this wave, MFMAs and softmax alike (its probabilities would all
  // be 0).  This leaves 10 of 16 wave-blocks of work in the clean quadrants'
  // diagonal tiles and 4 of 16 in the noisy-noisy ones (at S dividing 32).
  const int wr0 = q0 + 32 * __builtin_amdgcn_readfirstlane(w), wr1 = imin(q1, wr0 + 32);
  const PosWindow uw_n = wave_keys_visible(qh, HALF_NOISY, wr0, wr1, L, S);
  const PosWindow uw_c = wave_keys_visible(qh, HALF_CLEAN, wr0, wr1, L, S);

  // One FULL key tile.  The current K/V tiles and the buffers the next tile is
  // copied into are distinct restrict-qualified pointers: the alias scopes
  // this gives every LDS access let the compiler see that the copy in flight
  // cannot overwrite the tiles being read, so it does not wait for the copy
  // before the reads (the wait at the end of the step covers it).
  //
  // The copy of the next tile (K and V) is spread between the score MFMAs,
  // early enough in the step that the V part has landed by its end (issued
  // between the PV MFMAs instead, it made the end-of-step wait 2% of the
  // kernel).  A CU accepts vector memory requests at a limited rate, so a
  // burst of copies at the top of the step would stall the wave; spread out,
  // each request issues while MFMAs run.
  // The last step copies its own tile again (into the buffer nothing reads
  // afterwards), which keeps the step straight-line code.
  auto tile_step = [&](const char* __restrict__ kcur, const char* __restrict__ vcur, char* __restrict__ knxt,
                       char* __restrict__ vnxt, int t) __attribute__((always_inline)) {
    const int tn = imin(t + 1, T - 1);
    {
      f32x16 sacc[KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) sacc[kb][e] = 0.f;
      // S^T[key][query] = sum_d K[key][d] Q[query][d]
#pragma unroll
      for (int s = 0; s < DS; ++s)
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) sacc[kb] = mfma32(lds_rows<D>(kcur, ops.row_rel, s, kb), qreg[s], sacc[kb]);
      issue(tn, false, knxt);
      issue(tn, true, vnxt);
      // K operand reads four MFMAs ahead, the copies spread between the MFMAs
      pipeline_reads_and_copies<DS * KB, 4, 1, 2 * decltype(copy)::NI>();
      // (a FULL tile: every key is visible from every row, no test)
      // row maximum as a tree of three-input maxima (no serial chain)
      float m3[KB * 16 / 2];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int e = 0; e < 16; e += 2) m3[kb * 8 + e / 2] = fmaxf(sacc[kb][e], sacc[kb][e + 1]);
      float mx = tree_max<KB * 8>(m3);
      mx = halves_max(mx) * p.c;
      // move the reference only when this tile's max is far above it
      const bool grow = mx > m + RESCALE_SLACK;
      if (__any(grow)) {
        asm volatile("" ::: "memory");  // rare: keep the rescale out of the common path
        // lanes that do not grow keep factor 1 (their m may still be -inf);
        // a growing lane whose m is -inf gets exp2(-inf) = 0
        const float alpha = grow ? fast_exp2(m - mx) : 1.f;
        const float mnew = grow ? mx : m;
        lsum *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int e = 0; e < 16; ++e) oacc[db][e] *= alpha;
        m = mnew;
      }
      const float muse = (m == -INFINITY) ? 0.f : m;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) sacc[kb][e] = fast_exp2(sacc[kb][e] * p.c - muse);
      // the tile's row sum as a tree (no serial chain of 32 additions)
      lsum += tree_sum<KB>(sacc);
      bf16x8 pb[PC];
#pragma unroll
      for (int c = 0; c < PC; ++c) pb[c] = pack8(sacc[c >> 1], 8 * (c & 1));
      // O^T[d][query] += sum_key V^T[d][key] P^T[key][query]
#pragma unroll
      for (int c = 0; c < PC; ++c)
#pragma unroll
        for (int db = 0; db < DB; ++db) oacc[db] = mfma32(lds_tr<D>(vcur, ops.tr_rel0, ops.tr_rel1, c, db), pb[c], oacc[db]);
      pipeline_lds_reads<PC * DB, 4, 2>();  // V^T operand reads (two per MFMA) four MFMAs ahead
    }
  };
  // One 32-key block kb of a key tile, for the diagonal tiles: the same
  // arithmetic as a tile step restricted to those keys (masked by the window).
  // The next tile's copy is issued by the caller.
  auto block_step = [&](const char* __restrict__ kcur, const char* __restrict__ vcur, int kh, int k0, int kb)
                        __attribute__((always_inline)) {
    f32x16 sa;
#pragma unroll
    for (int e = 0; e < 16; ++e) sa[e] = 0.f;
#pragma unroll
    for (int s = 0; s < DS; ++s) sa = mfma32(lds_rows<D>(kcur, ops.row_rel, s, kb), qreg[s], sa);
    pipeline_lds_reads<DS, 4, 1>();
    const PosWindow win = kh == HALF_NOISY ? win_n : win_c;
    const unsigned span = (unsigned)(win.hi - win.lo);
    const int rel = k0 + 32 * kb + 4 * g2 - win.lo;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const unsigned pos = (unsigned)(rel + 8 * i + jj);
        sa[4 * i + jj] = pos < span ? sa[4 * i + jj] : -INFINITY;
      }
    float m3[8];
#pragma unroll
    for (int e = 0; e < 16; e += 2) m3[e / 2] = fmaxf(sa[e], sa[e + 1]);
    float mx = tree_max<8>(m3);
    mx = halves_max(mx) * p.c;
    const bool grow = mx > m + RESCALE_SLACK;
    if (__any(grow)) {
      asm volatile("" ::: "memory");
      const float alpha = grow ? fast_exp2(m - mx) : 1.f;
      const float mnew = grow ? mx : m;
      lsum *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[db][e] *= alpha;
      m = mnew;
    }
    const float muse = (m == -INFINITY) ? 0.f : m;
#pragma unroll
    for (int e = 0; e < 16; ++e) sa[e] = fast_exp2(sa[e] * p.c - muse);
    lsum += tree_sum<1>(&sa);
    const bf16x8 p0 = pack8(sa, 0), p1 = pack8(sa, 8);
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db] = mfma32(lds_tr<D>(vcur, ops.tr_rel0, ops.tr_rel1, 2 * kb, db), p0, oacc[db]);
#pragma unroll
    for (int db = 0; db < DB; ++db)
      oacc[db] = mfma32(lds_tr<D>(vcur, ops.tr_rel0, ops.tr_rel1, 2 * kb + 1, db), p1, oacc[db]);
  };
  auto step_buffers = [&](int t, char*& cur, char*& nxt) __attribute__((always_inline)) {
    cur = lds + (t & 1) * TILE;
    nxt = lds + ((t + 1) & 1) * TILE;
  };
  auto end_step = [&]() __attribute__((always_inline)) {
    compute_fence();
    wait_global_loads();  // this wave's part of the next tile has landed in LDS
    __syncthreads();      // ... for every wave, and every wave is done with this buffer
  };
  // The walk starts with the key tiles that are FULL for the whole query tile
  // (clean keys of earlier blocks); one loop with a single step body runs
  // them.  The remaining few tiles (the diagonal ones) run in a second loop
  // whose steps skip, per wave, the 32-key blocks none of its rows sees.
  // Keeping the two apart keeps the register assignment of the main loop
  // free of the copies that merging several step bodies in one loop costs.
  const int t_main = __builtin_amdgcn_readfirstlane(imin(T, fr.full_prefix(BN)));
  for (int t = 0; t < t_main; ++t) {
    char *cur, *nxt;
    step_buffers(t, cur, nxt);
    tile_step(cur, cur + 2 * TILE, nxt, nxt + 2 * TILE, t);
    end_step();
  }
  for (int t = t_main; t < T; ++t) {
    char *cur, *nxt;
    step_buffers(t, cur, nxt);
    int kh, j;
    kl.at(t, kh, j);
    const int k0 = j * BN;
    // (EMPTY tiles are never visited; were one visited, the window test of
    // PARTIAL tiles would mask all of it)
    const PosWindow uw = kh == HALF_NOISY ? uw_n : uw_c;
    const int tn = imin(t + 1, T - 1);
    issue(tn, false, nxt);
    issue(tn, true, nxt + 2 * TILE);
#pragma unroll 1
    for (int kb = 0; kb < KB; ++kb)  // (not unrolled: one block body in the loop)
      if (k0 + 32 * kb < uw.hi && k0 + 32 * kb + 32 > uw.lo) block_step(cur, cur + 2 * TILE, kh, k0, kb);
    end_step();
  }

  const float lt = halves_sum(lsum);
  if (qvalid) {
    const float inv = 1.f / lt;
    bf16* op = p.O + (qbase + prow) * D + 4 * g2;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        st_bf16x4(op + db * 32 + 8 * i, oacc[db][4 * i] * inv, oacc[db][4 * i + 1] * inv,
                  oacc[db][4 * i + 2] * inv, oacc[db][4 * i + 3] * inv);
    if (g2 == 0) p.LSE[qbase + prow] = (m + log2f(lt)) * LN2;
  }
}

template <int D>
hipError_t launch_fwd_d(const Shape& s, const void* Q, const void* K, const void* V, void* O,
                        float* LSE, hipStream_t st, LaunchEvents ev) {
  FwdParams p;
  p.Q = static_cast<const bf16*>(Q);
  p.K = static_cast<const bf16*>(K);
  p.V = static_cast<const bf16*>(V);
  p.O = static_cast<bf16*>(O);
  p.LSE = LSE;
  p.seq = s.seq;
  p.L = s.L;
  p.S = s.S;
  p.Hq = s.Hq;
  p.Hkv = s.Hkv;
  p.G = s.G;
  p.nQT = cdiv(s.L, FWD_BM);
  p.nbh = s.B * s.Hq;
  p.c = s.scale * LOG2E;
  const dim3 grid(2 * p.nQT * p.nbh);
  hipExtLaunchKernelGGL(fwd_kernel<D>, grid, dim3(256), 0, st, ev.start, ev.stop, 0, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_fwd(const Shape& s, const void* Q, const void* K, const void* V, void* O,
                      float* LSE, hipStream_t st, LaunchEvents ev) {
  if (s.D == 128) return launch_fwd_d<128>(s, Q, K, V, O, LSE, st, ev);
  return launch_fwd_d<64>(s, Q, K, V, O, LSE, st, ev);
}

}  // namespace bd
