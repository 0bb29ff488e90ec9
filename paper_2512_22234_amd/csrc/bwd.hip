// Backward pass of block-diffusion masked attention for gfx950: the
// vector-Jacobian product of softmax attention under the mask of Eq. 1 / Eq. 2
// (DiRL Section 4.1), with no floating-point atomics, so results are bitwise
// reproducible.
//
//   Delta = rowsum(dO * O), lse2 = LSE * log2(e)        (dq prologue)
//   P     = exp2(scale*log2(e) * Q K^T - lse2) on visible pairs
//   dV    = P^T dO,  dP = dO V^T,  dS = P * (dP - Delta)
//   dQ    = scale dS K                                  (dq, query-tile major; runs first)
//   dK    = scale dS^T Q                                (dkdv, key-tile major)
//
// dkdv: a workgroup owns a (batch, KV head, 128-key tile) and walks the query
// heads of the GQA group and the 32-row query tiles that can see the key tile
// (the exact tile classification gives the list).  Its eight waves split the
// work by role: four producers compute S = Q K^T and dP = dO V^T (each lane
// owns one key column), then P and dS, and pass P and dS through LDS as bf16
// MFMA operands; four consumers, one on each SIMD beside a producer, keep dK
// and dV and accumulate dV^T = dO^T P and dK^T = Q^T dS, whose A operands come
// from the Q and dO tiles through the transposing LDS read.  Work per clean
// key tile shrinks linearly with its position, so each clean tile's walk is
// split into parts (two, or four when the heaviest half-walk would outlast the
// average work of a CU) run by as many workgroups.  Every part but the last to
// finish leaves its float32 sums in the workspace; the last adds all of them,
// its own included, in part order and writes dK/dV, so the result does not
// depend on which part finishes when.  Noisy key tiles (seen only by their
// own block's noisy queries) are done by one workgroup each.
//
// dq: a workgroup owns a (batch, query head, 128-row query tile) like the
// forward; scores are S^T = K Q^T (lane = query) and dQ^T = K^T dS^T with K^T
// read from the K tile through the transposing LDS read.  Its prologue also
// computes Delta and lse2 of its rows for the dK/dV kernel, and the kernel
// clears the counters with which the dK/dV kernel pairs its split walks.
//
// Tiles are copied into LDS asynchronously with buffer loads to LDS, ahead of
// the step that reads them.
#include "device.hpp"
#include "kernels.hpp"

namespace bd {
namespace {

// ----------------------------------------------------------------------------
struct DkvParams {
  const bf16* Q;
  const bf16* K;
  const bf16* V;
  const bf16* dO;
  const float* rs;  // (lse2, delta) per query row
  bf16* dK;
  bf16* dV;
  float* part;  // [nsplit - 1 arrival slots][tile slots][4 consumer waves][32 x 16 bytes per lane]: unscaled sums of the parts of a clean key tile's walk that did not finish last
  int* pair;    // per (clean key tile, key group): DKV_PAIR_INTS counters (arrivals, published, slot owners), zeroed by the dq kernel
  SeqLayout seq;
  size_t tile_slots;               // regions of one arrival slot of `part`: clean key tiles of every sequence and KV head
  int L, S, Hq, Hkv, G, nKT, nkv;  // L: the (maximum) sequence length; nkv: sequences x KV heads
  float c;      // scale * log2(e)
  float scale;
};

template <int D>
struct DkvSmem {
  static constexpr int BM = DKV_BM;
  static constexpr uint32_t TILE = BM * D * 2;  // bytes per swizzled tile
  // one contiguous region per buffer: Q tile, dO tile, (lse2, delta) per row
  static constexpr uint32_t DO_OFF = TILE, RS_OFF = 2 * TILE;
  static constexpr uint32_t BUF = 2 * TILE + 8 * BM;  // a multiple of 256 bytes
  static constexpr int NBUF = 5;                      // copies run three steps ahead
  // P and dS of one key group (32 keys x BM queries), as the bf16 B operands
  // of the consumer's MFMAs: operand h of P at 2h KiB, of dS at (2h+1) KiB,
  // 16 bytes per lane.
  static constexpr uint32_t XGRP = 4 * BM * 32;
  static constexpr uint32_t XBUF = 4 * XGRP;
  static_assert(BUF % 256 == 0 && XBUF % 256 == 0, "operand addressing needs 256-byte aligned tiles");
  static_assert(BM == 32, "one 32-query block per step");
  // Noisy key tiles whose key groups each see one 32-query block (S divides
  // 32): two sets of the four query tiles under the key tile (one query head
  // each) and one P/dS buffer.
  static constexpr int NBUF_NOISY = 8;
  static constexpr uint32_t CLEAN_BYTES = NBUF * BUF + 2 * XBUF, NOISY_BYTES = NBUF_NOISY * BUF + XBUF;
  alignas(256) char mem[CLEAN_BYTES > NOISY_BYTES ? CLEAN_BYTES : NOISY_BYTES];
  // clean key tiles: query-tile buffer i, P/dS buffer i
  __device__ char* buf(int i) { return mem + i * BUF; }
  __device__ char* x(int i) { return mem + NBUF * BUF + i * XBUF; }
  // noisy key tiles: query tile u (of four) of set `set`, and the P/dS buffer
  __device__ char* nbuf(int set, int u) { return mem + (4 * set + u) * BUF; }
  __device__ char* nx() { return mem + NBUF_NOISY * BUF; }
};

// Workgroup of eight waves on one (batch, KV head, 128-key tile).  Waves w and
// w + 4 run on the same SIMD and share the 32 keys k0 + 32 (w % 4) + [0, 32):
//   producer (w < 4): K and V rows of its keys in registers; S and dP of one
//     32-query block, then P and dS, written to LDS as bf16 operands.  It is
//     software-pipelined: step t computes P and dS of block t while the MFMAs
//     of S and dP of block t + 1 run;
//   consumer (w >= 4): the dK and dV accumulators; per step the two products
//     of the block the producer finished one step earlier, and the copy of the
//     query tile three steps ahead.
// A producer's softmax arithmetic thus runs beside MFMAs (its own and its
// consumer's) on the same SIMD, and each role fits the register budget of two
// waves per SIMD.  One barrier per step; it drains LDS operations only, so the
// copies issued in a step stay in flight across it.  In step t the query-tile buffers
// hold tiles t - 1 (consumer), t and t + 1 (producer), t + 2 (landed or
// landing) and t + 3 (being copied); the P/dS buffers steps t and t - 1.
template <int D, int NSPLIT>
__global__ __launch_bounds__(512, 1) void dkdv_kernel(DkvParams p) {
  constexpr int BM = DKV_BM, BN = DKV_BN;
  constexpr int DS = D / 16, DB = D / 32;
  using Smem = DkvSmem<D>;
  __shared__ Smem sm;

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kg = w & 3;  // key group
  const int l32 = lane & 31, g2 = lane >> 5;

  // Items: clean key tiles, most work first, each as nsplit parts of its
  // walk; then noisy key tiles, one item each.  A clean key tile at k0 is seen
  // by about 2 (L - k0) queries, so the work of a tile is set by how many
  // tiles of its sequence follow it.  Fixed length: item rank r is tile r,
  // consecutive workgroups being different KV heads and sequences.  Packed
  // sequences: one ranking of all sequences' key tiles by the tiles from each
  // to its sequence's end, largest first (the grid is sized by a bound on
  // their count); the parts and KV heads of one tile are consecutive items.
  const int id = blockIdx.x;
  constexpr int nsplit = NSPLIT;
  int b, hk, split, j;
  bool clean;
  int pc0 = 0, plen = 0;  // packed: the sequence's first token and length
  size_t tslot;           // region of the partial sums of this key tile (clean items)
  if (p.seq.cu == nullptr) {
    const int rank = id / p.nkv;
    const int grp0 = id - rank * p.nkv;  // b * Hkv + hk
    const int crank = rank / nsplit;
    clean = rank < nsplit * p.nKT;
    split = clean ? rank - crank * nsplit : 0;
    b = grp0 / p.Hkv;
    hk = grp0 - b * p.Hkv;
    j = clean ? crank : rank - nsplit * p.nKT;
    tslot = (size_t)j * p.nkv + grp0;
  } else {
    const int n = p.nkv / p.Hkv;
    const int nclean = nsplit * p.Hkv * packed_rows(p.seq.cu, n, BN);
    int r;
    clean = id < nclean;
    if (clean) {
      r = id / (nsplit * p.Hkv);
      const int q = id - r * nsplit * p.Hkv;
      split = q / p.Hkv;
      hk = q - split * p.Hkv;
    } else {
      r = (id - nclean) / p.Hkv;
      hk = id - nclean - r * p.Hkv;
      split = 0;
    }
    int i, nt;
    if (!packed_row(p.seq.cu, n, p.nKT, BN, r, b, i, nt, pc0, plen)) return;  // past the last tile
    j = nt - 1 - i;
    tslot = (size_t)r * p.Hkv + hk;
  }
  const int kh = clean ? HALF_CLEAN : HALF_NOISY;
  const int grp = b * p.Hkv + hk;
  // sequence b: its length and where its rows lie
  int L;
  size_t qrow0, krow0, hrows;
  if (p.seq.cu == nullptr) p.seq.get(b, p.L, p.Hq, p.Hkv, L, qrow0, krow0, hrows);
  else p.seq.get_packed(pc0, plen, L, qrow0, krow0, hrows);
  if (j * BN >= L) return;  // (fixed length: never)
  // (a sequence shorter than S is one block: every formula below gives
  // the S = L mask then)
  const int S = p.S;
  const int N = 2 * L;
  const int k0 = j * BN, k1 = imin(L, k0 + BN);
  const size_t khead = krow0 + hk * hrows;  // row of this KV head's position 0 in K, V, dK, dV

  const int kk = k0 + kg * 32 + l32;  // this lane's key (local to its half)
  const bool kvalid = kk < k1;
  const int kblock0 = kvalid ? (kk / S) * S : 0;
  const size_t krow = khead + kh * L + kk;

  // A noisy key group is seen only by the noisy queries of its own blocks;
  // when S divides 32 those are exactly the 32 queries at the same positions,
  // so each producer scores its own query block and a noisy key tile takes one
  // step per query head (a walk over the four query tiles would leave three
  // of the four producers without a visible pair in every step).
  const bool noisy_diag = !clean && 32 % S == 0;
  const QueryWalk wk = query_walk(kh, j, split, nsplit, L, S, BM, BN, p.G);
  const int T = wk.steps();
  const int steps = T > 0 ? T + 1 : 0;  // the consumer trails the producer by one step
  const WalkPos first = wk.first(), last = wk.last();
  const LdsOperands<D> ops(lane);

  if (w < 4) {
    // ---------------------------------------------------------------- producer
    bf16x8 kreg[DS], vreg[DS];
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      kreg[s] = kvalid ? *reinterpret_cast<const bf16x8*>(p.K + krow * D + 16 * s + 8 * g2) : zero_bf16x8();
      vreg[s] = kvalid ? *reinterpret_cast<const bf16x8*>(p.V + krow * D + 16 * s + 8 * g2) : zero_bf16x8();
    }
    // S[q][key] = sum_d Q[q][d] K[key][d];  dP[q][key] = sum_d dO[q][d] V[key][d]
    auto scores = [&](const char* __restrict__ bt, f32x16& sacc, f32x16& dpacc) __attribute__((always_inline)) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        sacc[e] = 0.f;
        dpacc[e] = 0.f;
      }
#pragma unroll
      for (int s = 0; s < DS; ++s) {
        sacc = mfma32(lds_rows<D>(bt, ops.row_rel, s, 0), kreg[s], sacc);
        dpacc = mfma32(lds_rows<D>(bt + Smem::DO_OFF, ops.row_rel, s, 0), vreg[s], dpacc);
      }
    };
    // P = exp2(c S - lse2), dS = P (dP - delta) of block t, into xw as bf16
    // operands; query q0 + offset sees this lane's key iff
    // win.lo <= q0 + offset < win.hi (FULL tiles: every query does).
    auto softmax_grad = [&](const char* __restrict__ bt, char* __restrict__ xw, f32x16& sacc, f32x16& dpacc,
                            int rel, unsigned span, auto masked) __attribute__((always_inline)) {
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int rr = 8 * i4 + 4 * g2;  // rows rr .. rr + 3 of this lane's accumulator slots
        const f32x4 a = *reinterpret_cast<const f32x4*>(bt + Smem::RS_OFF + 8 * rr);
        const f32x4 z = *reinterpret_cast<const f32x4*>(bt + Smem::RS_OFF + 8 * rr + 16);
        const float l4[4] = {a[0], a[2], z[0], z[2]}, d4[4] = {a[1], a[3], z[1], z[3]};
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int e = 4 * i4 + jj;
          float pv = fast_exp2(sacc[e] * p.c - l4[jj]);
          if constexpr (decltype(masked)::value) pv = (unsigned)(rel + 8 * i4 + jj) < span ? pv : 0.f;
          dpacc[e] = pv * (dpacc[e] - d4[jj]);
          sacc[e] = pv;
        }
      }
      char* xg = xw + kg * Smem::XGRP + 16 * lane;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        *reinterpret_cast<bf16x8*>(xg + 2 * h * 1024) = pack8(sacc, 8 * h);
        *reinterpret_cast<bf16x8*>(xg + (2 * h + 1) * 1024) = pack8(dpacc, 8 * h);
      }
    };
    // Step t: scores of block t + 1 into (sn, dn) beside the softmax gradient
    // of block t from (sc, dc).  Past the last block the buffer of t + 1 holds
    // a repeated tile: its scores are computed and never used.  The per-step
    // bookkeeping is kept to a few scalar instructions: the FULL test is two
    // comparisons against per-workgroup bounds, the visibility windows of
    // both halves are computed once, and the buffers rotate by offset.
    const FullRange fr = full_range_vs_key_tile(kh, k0, k1, L, S, BN);
    const PosWindow win_n = queries_seeing(kh, HALF_NOISY, kblock0, L, S, kvalid);
    const PosWindow win_c = queries_seeing(kh, HALF_CLEAN, kblock0, L, S, kvalid);
    WalkPos cur = first;
    uint32_t bcur = 0;  // byte offset of tile t's buffer (tile t + 1's follows, modulo NBUF)
    // Clean key tiles: blocks in which no query sees any key of this group
    // (on the diagonal, at the end of the walk) are skipped: no scores, and no
    // P or dS for the consumers, which skip them too.  (The queries seeing a
    // clean key group also see every earlier group's keys, which the
    // consumers rely on.)  The steps before the first such block run without
    // the tests, so that they keep their schedule: the tests split a step's
    // code into pieces the scores' MFMAs cannot interleave across.
    const KeyGroupSight sight(kh, k0 + 32 * kg, k1, L, S);
    const int U = clean ? first_unseen_step(wk, sight, BM, L) : T;  // blocks [0, U) are seen
    bool vis = U > 0;                                               // block t is seen
    auto step = [&](int t, f32x16& sc, f32x16& dc, f32x16& sn, f32x16& dn, auto tested)
                    __attribute__((always_inline)) {
      const int qh = cur.qh, q0 = cur.tile(wk) * BM;
      cur.next(wk);
      const uint32_t bnext = bcur == (Smem::NBUF - 1) * Smem::BUF ? 0u : bcur + Smem::BUF;
      const char* bt = sm.mem + bcur;
      const char* bn = sm.mem + bnext;
      bcur = bnext;
      char* xw = sm.x(t & 1);
      // (EMPTY tiles are never visited; the window test would mask all of one)
      if constexpr (!decltype(tested)::value) {
        if (fr.full(qh, q0, BM)) {
          scores(bn, sn, dn);
          softmax_grad(bt, xw, sc, dc, 0, 0u, Flag<false>());
        } else {
          const PosWindow win = qh == HALF_NOISY ? win_n : win_c;
          scores(bn, sn, dn);
          softmax_grad(bt, xw, sc, dc, q0 + 4 * g2 - win.lo, (unsigned)(win.hi - win.lo), Flag<true>());
        }
      } else {
        const bool vis_t = vis;
        vis = !clean || sight.sees(cur.qh, cur.tile(wk) * BM, BM, L);  // block t + 1 (past the end: unused)
        // (each case one straight run of code)
        if (fr.full(qh, q0, BM)) {
          if (vis) {
            scores(bn, sn, dn);
            softmax_grad(bt, xw, sc, dc, 0, 0u, Flag<false>());
          } else {
            softmax_grad(bt, xw, sc, dc, 0, 0u, Flag<false>());
          }
        } else {
          const PosWindow win = qh == HALF_NOISY ? win_n : win_c;
          const int rel = q0 + 4 * g2 - win.lo;
          const unsigned span = (unsigned)(win.hi - win.lo);
          if (vis && vis_t) {
            scores(bn, sn, dn);
            softmax_grad(bt, xw, sc, dc, rel, span, Flag<true>());
          } else if (vis) {
            scores(bn, sn, dn);
          } else if (vis_t) {
            softmax_grad(bt, xw, sc, dc, rel, span, Flag<true>());
          }
        }
      }
    };
    if (noisy_diag) {
      // Per query head g: S and dP of this key group against query block kg
      // of set g % 2, then P and dS (visibility window per element), written
      // for the consumers; no software pipeline (one step per head).
      const unsigned span = (unsigned)(win_n.hi - win_n.lo);
      const int rel = k0 + 32 * kg + 4 * g2 - win_n.lo;
      for (int g = 0; g < p.G; ++g) {
        barrier_lds_only();  // set g % 2 has landed; the consumers are done with the P/dS buffer
        const char* bt = sm.nbuf(g & 1, kg);
        f32x16 sc, dc;
        scores(bt, sc, dc);
        softmax_grad(bt, sm.nx(), sc, dc, rel, span, Flag<true>());
        barrier_lds_only();  // P and dS are written
      }
      return;
    }
    f32x16 sA, dA, sB, dB;
    __syncthreads();  // the first three query tiles are in LDS
    if (vis) scores(sm.mem, sA, dA);
    // steps alternate the two accumulator pairs (unrolled by two, no copies);
    // untested steps t need blocks t and t + 1 seen (an even number of them)
    const int E = imax(0, U - 1) & ~1;
    for (int t = 0; t < E; t += 2) {
      step(t, sA, dA, sB, dB, Flag<false>());
      barrier_lds_only();
      step(t + 1, sB, dB, sA, dA, Flag<false>());
      barrier_lds_only();
    }
    for (int t = E; t < T; t += 2) {
      step(t, sA, dA, sB, dB, Flag<true>());
      barrier_lds_only();
      if (t + 1 < T) {
        step(t + 1, sB, dB, sA, dA, Flag<true>());
        barrier_lds_only();
      }
    }
    if (T > 0) barrier_lds_only();  // the consumer's last step
  } else {
    // ---------------------------------------------------------------- consumer
    // Consumer c = w - 4 owns one tensor (dV for c < 2, dK for c >= 2) of the
    // 64 keys k0 + 64 (c % 2) + [0, 64), i.e. key groups 2 (c % 2) and
    // 2 (c % 2) + 1: every dO^T or Q^T operand it reads serves two MFMAs.
    const int c = w - 4;
    const bool isdk = c >= 2;
    const int kc0 = k0 + 64 * (c & 1);
    const TileCopy<D, BM, 256> copy(tid - 256);
    constexpr int NC = 2 * decltype(copy)::NI + 1;  // vector-memory instructions per query-tile copy
    // Q, dO and (lse2, delta) of one query tile.  The four waves copy the
    // row pairs each (the same data), so every wave issues NC instructions.
    // Addresses: the group's first query head is fixed, so a step adds one
    // row offset (head g, packed row row0) to three base pointers.
    const size_t g0row = qrow0 + (size_t)hk * p.G * hrows;  // first row of the group's first head
    const bf16* const qg = p.Q + g0row * D;
    const bf16* const dog = p.dO + g0row * D;
    const float* const rsg = p.rs + 2 * g0row;
    auto issue = [&](WalkPos wp, char* dst) {
      const int row0 = wp.qh * L + wp.tile(wk) * BM;
      const size_t r = (size_t)wp.g * hrows + row0;  // row within the group's heads
      const int left = N - row0;                 // rows of this head from row0 on
      copy.issue_rows(qg + r * D, left, dst);
      copy.issue_rows(dog + r * D, left, dst + Smem::DO_OFF);
      async_load_row_floats(rsg + 2 * r, 2 * left, 0, reinterpret_cast<float*>(dst + Smem::RS_OFF), lane);
    };
    f32x16 acc[2][DB];  // [key group of 32][feature block of 32]
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[ks][db][e] = 0.f;
    const uint32_t aoff = isdk ? 0u : Smem::DO_OFF;  // A operand: Q^T or dO^T
    const int xsel = isdk ? 1 : 0;                   // B operand: dS or P
    if (noisy_diag) {
      // The four noisy query tiles under the key tile, for query head g,
      // into set s (two sets: head g + 1 lands while head g is computed).
      auto issue_head = [&](int g, int set) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int row0 = k0 + 32 * u;  // noisy half: local position = row
          const size_t r = (size_t)g * hrows + row0;
          const int left = N - row0;
          char* dst = sm.nbuf(set, u);
          copy.issue_rows(qg + r * D, left, dst);
          copy.issue_rows(dog + r * D, left, dst + Smem::DO_OFF);
          async_load_row_floats(rsg + 2 * r, 2 * left, 0, reinterpret_cast<float*>(dst + Smem::RS_OFF), lane);
        }
      };
      issue_head(0, 0);
      if (p.G > 1) issue_head(1, 1);
      for (int g = 0; g < p.G; ++g) {
        // set g % 2 has landed in this wave's part (before head 0 the copy of
        // head 1 may still be in flight; later the copy in flight is head g's,
        // issued in the previous iteration) ...
        if (g == 0 && p.G > 1) wait_global_loads_but<4 * NC>();
        else wait_global_loads();
        barrier_lds_only();  // ... and in every wave's
        // set (g + 1) % 2 held head g - 1, which everyone is done with
        if (g >= 1 && g + 1 < p.G) issue_head(g + 1, (g + 1) & 1);
        barrier_lds_only();  // the producers have written P and dS of head g
        // key group 2 (c % 2) + ks saw query block 2 (c % 2) + ks of the set
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const int grp4 = 2 * (c & 1) + ks;
          const char* bc = sm.nbuf(g & 1, grp4);
          bf16x8 xb[2];
#pragma unroll
          for (int h = 0; h < 2; ++h)
            xb[h] = *reinterpret_cast<const bf16x8*>(sm.nx() + grp4 * Smem::XGRP + 16 * lane + (2 * h + xsel) * 1024);
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int db = 0; db < DB; ++db)
              acc[ks][db] = mfma32(lds_tr<D>(bc + aoff, ops.tr_rel0, ops.tr_rel1, h, db), xb[h], acc[ks][db]);
        }
      }
    } else {
    // tiles 0, 1 and 2 (the last tile again past the end); cp then points at tile 3
    WalkPos cp = first;
    if (T > 0) {
#pragma unroll
      for (int u = 0; u < 3; ++u) {
        issue(u < T ? cp : last, sm.buf(u));
        cp.next(wk);
      }
    }
    wait_global_loads();
    __syncthreads();

    // Step t: the products of the block of step t - 1, then the copy of tile
    // t + 3 (the last tile again past the end, into a buffer nothing reads
    // any more, so every step issues the same copies).  The buffers read and
    // the one written are distinct restrict-qualified pointers, so the
    // compiler does not wait for the copy in flight before the reads.
    //   dV^T[d][key] += sum_q dO^T[d][q] P[q][key]   (dV consumers)
    //   dK^T[d][key] += sum_q Q^T[d][q] dS[q][key]   (dK consumers)
    // The products of key group 2 (c % 2) + ks skip the blocks its producer
    // skipped (clean key tiles; a block the second group is seen in is seen by
    // the first too).  Blocks before the first one the second group is not
    // seen in need no test.
    const KeyGroupSight sight0(kh, kc0, k1, L, S), sight1(kh, kc0 + 32, k1, L, S);
    const int U1 = clean ? first_unseen_step(wk, sight1, BM, L) : T;  // blocks [0, U1) are seen by both
    WalkPos cc = U1 < T ? wk.at(U1) : first;                          // block of step t - 1 (tested steps)
    auto products = [&](const char* __restrict__ bc, const char* __restrict__ xr, auto use0, auto use1)
                        __attribute__((always_inline)) {
      constexpr bool u0 = decltype(use0)::value, u1 = decltype(use1)::value;
      bf16x8 xb[2][2];  // [key group][16-query half]
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          if (ks == 0 ? u0 : u1)
            xb[ks][h] = *reinterpret_cast<const bf16x8*>(xr + (2 * (c & 1) + ks) * Smem::XGRP + 16 * lane +
                                                         (2 * h + xsel) * 1024);
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const bf16x8 a = lds_tr<D>(bc + aoff, ops.tr_rel0, ops.tr_rel1, h, db);
          if constexpr (u0) acc[0][db] = mfma32(a, xb[0][h], acc[0][db]);
          if constexpr (u1) acc[1][db] = mfma32(a, xb[1][h], acc[1][db]);
        }
    };
    auto consume = [&](const char* __restrict__ bc, const char* __restrict__ xr, char* __restrict__ bn, int t,
                       auto tested) __attribute__((always_inline)) {
      if constexpr (!decltype(tested)::value) {
        if (t > 0) products(bc, xr, Flag<true>(), Flag<true>());
        issue(t + 3 < T ? cp : last, bn);
      } else {
        // (t > 0; each case one straight run of code)
        const int qc = cc.tile(wk) * BM;
        const bool v0 = !clean || sight0.sees(cc.qh, qc, BM, L), v1 = !clean || sight1.sees(cc.qh, qc, BM, L);
        cc.next(wk);
        if (v1) {
          products(bc, xr, Flag<true>(), Flag<true>());
          issue(t + 3 < T ? cp : last, bn);
        } else if (v0) {
          products(bc, xr, Flag<true>(), Flag<false>());
          issue(t + 3 < T ? cp : last, bn);
        } else {
          issue(t + 3 < T ? cp : last, bn);
        }
      }
    };
    uint32_t bcons = (Smem::NBUF - 1) * Smem::BUF;  // buffer of tile t - 1
    uint32_t bcopy = 3 * Smem::BUF;                  // buffer tile t + 3 is copied into
    auto consumer_step = [&](int t, auto tested) __attribute__((always_inline)) {
      consume(sm.mem + bcons, sm.x((t + 1) & 1), sm.mem + bcopy, t, tested);
      bcons = bcons == (Smem::NBUF - 1) * Smem::BUF ? 0u : bcons + Smem::BUF;
      bcopy = bcopy == (Smem::NBUF - 1) * Smem::BUF ? 0u : bcopy + Smem::BUF;
      if (t + 3 < T) cp.next(wk);
      compute_fence();
      wait_global_loads_but<NC>();  // tile t + 2 has landed (the copy issued this step may not have)
      barrier_lds_only();           // ... in every wave's part; the copy in flight stays in flight
    };
    const int E = imin(steps, U1 + 1);  // steps whose block t - 1 < U1
    for (int t = 0; t < E; ++t) consumer_step(t, Flag<false>());
    for (int t = E; t < steps; ++t) consumer_step(t, Flag<true>());
    }
    wait_global_loads();  // no copy may still be writing LDS when the workgroup ends

    const float sc = isdk ? p.scale : 1.f;
    bf16* const outp = isdk ? p.dK : p.dV;
    const size_t orow = khead + kh * L;  // first row of this KV head's half
    if (clean) {
      // The parts of this key tile's walk meet here, per consumer wave.  Each
      // takes an arrival slot from the counter; every part but the last
      // stores its float32 sums in its slot, records its part index for that
      // slot (slots past the first; the part not found there is in slot 0)
      // and then counts itself as published.  The last waits until every other
      // part has published (each has arrived, so it is running and only
      // stores), then adds the nsplit sums in part order, its own in place,
      // and writes its tensor: the result is the same whichever part arrives
      // when.  The sums are stored unscaled and dK is scaled after the
      // addition, so no multiply-add can fuse one part's product into the sum.
      //
      // The sums, slot owners and counters are written and read with
      // device-scope (sc1) accesses, which the L2 of one XCD does not hold
      // back from another, and the sums and owner are complete (vmcnt) before
      // the published count moves.  Cache-wide release/acquire fences would
      // instead write back and invalidate the whole L2 under the workgroups
      // still running.
      //
      // The sums travel in the register order of the consumer waves (the
      // same in every part): accumulator quad u = (ks DB + db) 4 + i of lane
      // l at byte 1024 u + 16 l of this wave's 32 KiB region, so each store
      // or load instruction moves 1 KiB of consecutive bytes (a layout by key
      // row would write 32-byte pieces of 32 rows per instruction).
      int* cnt = p.pair + DKV_PAIR_INTS * ((j * p.nkv + grp) * 4 + c);
      int* published = cnt + 1;
      int* owner = cnt + 2;  // part index of the sums in each arrival slot
      auto slot_buffer = [&](int a) __attribute__((always_inline)) {
        const float* pbase = p.part + (((size_t)a * p.tile_slots + tslot) * 4 + c) * (BN / 2) * D;
        return make_buffer(pbase, (uint32_t)((BN / 2) * D * 4));
      };
      const uint32_t loff = 16 * (uint32_t)lane;
      constexpr int SC1 = 16;  // cache-policy bit: device scope
      int order = 0;
      if (lane == 0) order = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      order = __builtin_amdgcn_readfirstlane(order);
      if (order < nsplit - 1) {
        const __amdgpu_buffer_rsrc_t pr = slot_buffer(order);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const f32x4 v = {acc[ks][db][4 * i], acc[ks][db][4 * i + 1], acc[ks][db][4 * i + 2],
                               acc[ks][db][4 * i + 3]};
              __builtin_amdgcn_raw_buffer_store_b128(v, pr, loff + 1024 * ((ks * DB + db) * 4 + i), 0, SC1);
            }
        // (slot 0's owner is never read: a part missing from slots 1 .. is in slot 0)
        if (order > 0 && lane == 0) __hip_atomic_store(owner + order, split, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the sums and the owner have reached device scope
        if (lane == 0) __hip_atomic_fetch_add(published, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
      }
      // Bounded wait (every other part is past its last step and only stores
      // its sums); the bound only guarantees that the wave always ends.
      int seen = 0;
      for (int spin = 0; spin < (1 << 22); ++spin) {
        seen = __builtin_amdgcn_readfirstlane(
            __hip_atomic_load(published, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
        if (seen == nsplit - 1) break;
        __builtin_amdgcn_s_sleep(2);
      }
      asm volatile("" ::: "memory");
      if (seen != nsplit - 1) {
        // Some part's sums were never published: the result would be wrong,
        // so this wave's keys get NaN instead of a plausible value.
        const float nan = __builtin_nanf("");
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const int key = kc0 + 32 * ks + l32;
          if (key < k1) {
            bf16* op = outp + (orow + key) * D + 4 * g2;
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
              for (int i = 0; i < 4; ++i) st_bf16x4(op + db * 32 + 8 * i, nan, nan, nan, nan);
          }
        }
        return;
      }
      // the part whose sums arrival slots 1 and 2 hold (-1: no such slot; two
      // parts have none)
      int own_of[3] = {-1, -1, -1};
#pragma unroll
      for (int a = 1; a < nsplit - 1; ++a)
        own_of[a] = __builtin_amdgcn_readfirstlane(
            __hip_atomic_load(owner + a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
      // arrival slot of part q: slot 0 unless slot 1 or 2 holds it (also for
      // this part, whose sums are its own: a valid slot, so that a load the
      // compiler issues anyway stays in bounds)
      auto slot_of = [&](int q) __attribute__((always_inline)) {
        return q == own_of[1] ? 1 : q == own_of[2] ? 2 : 0;
      };
      // Output rows kc0 .. k1 - 1 of this tensor through a buffer descriptor
      // that ends at k1: stores of keys past a ragged end fall outside it and
      // are dropped, so no branch separates the loads of one group of
      // accumulator quads from the next and the loads can be issued together.
      const __amdgpu_buffer_rsrc_t ob =
          make_buffer(outp + (orow + kc0) * D, (uint32_t)(imax(0, imin(BN / 2, k1 - kc0)) * D * 2));
      // groups of GQ accumulator quads: the other parts' sums of a group are
      // loaded together (nsplit - 1 of them per quad)
      constexpr int GQ = nsplit == 2 ? 8 : 4;
#pragma unroll
      for (int g0 = 0; g0 < 2 * DB * 4; g0 += GQ) {
        f32x4 oth[nsplit][GQ];
#pragma unroll
        for (int q = 0; q < nsplit; ++q)
#pragma unroll
          for (int u = 0; u < GQ; ++u)
            if (q != split)
              oth[q][u] = __builtin_amdgcn_raw_buffer_load_b128(slot_buffer(slot_of(q)), loff + 1024 * (g0 + u), 0, SC1);
#pragma unroll
        for (int u = 0; u < GQ; ++u) {
          const int qd = g0 + u, ks = qd / (4 * DB), db = (qd / 4) % DB, i = qd % 4;
          const f32x4 own = {acc[ks][db][4 * i], acc[ks][db][4 * i + 1], acc[ks][db][4 * i + 2], acc[ks][db][4 * i + 3]};
          f32x4 tot = own;
#pragma unroll
          for (int q = 0; q < nsplit; ++q) {
            const f32x4 x = q == split ? own : oth[q][u];
            tot = q == 0 ? x : tot + x;
          }
          bf16x4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = (bf16)(tot[e] * sc);
          typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
          __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, o), ob,
                                                (uint32_t)(((32 * ks + l32) * D + 32 * db + 8 * i + 4 * g2) * 2), 0, 0);
        }
      }
    } else {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int key = kc0 + 32 * ks + l32;
        if (key < k1) {
          bf16* op = outp + (orow + key) * D + 4 * g2;
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              st_bf16x4(op + db * 32 + 8 * i, acc[ks][db][4 * i] * sc, acc[ks][db][4 * i + 1] * sc,
                        acc[ks][db][4 * i + 2] * sc, acc[ks][db][4 * i + 3] * sc);
        }
      }
    }
  }
}

// ----------------------------------------------------------------------------
struct DqParams {
  const bf16* Q;
  const bf16* K;
  const bf16* V;
  const bf16* dO;
  const bf16* O;
  const float* LSE;
  float* rs;  // out: (lse2, delta) per query row, for the dK/dV kernel
  int* pair;  // dK/dV pairing counters, cleared here
  int npair;
  bf16* dQ;
  SeqLayout seq;
  int L, S, Hq, Hkv, G, nQT, nbh;
  float c;
  float scale;
};

template <int D>
struct DqSmem {
  static constexpr int BN = DQ_BN;
  static constexpr uint32_t TILE = BN * D * 2;  // bytes per swizzled tile
  bf16 k[2][BN * D];  // byte offset buf * TILE
  bf16 v[2][BN * D];  // byte offset (2 + buf) * TILE
};

template <int D>
__global__ __launch_bounds__(256, 2) void dq_kernel(DqParams p) {
  constexpr int BM = DQ_BM, BN = DQ_BN;
  constexpr int DS = D / 16, DB = D / 32, KB = BN / 32, PC = BN / 16;
  constexpr uint32_t TILE = DqSmem<D>::TILE;
  __shared__ DqSmem<D> sm;
  char* lds = reinterpret_cast<char*>(&sm);

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, g2 = lane >> 5;

  const int id = blockIdx.x;
  for (int i = id * 256 + tid; i < p.npair; i += gridDim.x * 256) p.pair[i] = 0;
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

  const int r = q0 + w * 32 + l32;
  const bool qvalid = r < q1;
  const int qblock0 = qvalid ? (r / S) * S : 0;
  const int prow = qh * L + r;
  const size_t qrow = qrow0 + hq * hrows + prow;

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
  auto issue = [&](int t, char* kdst, char* vdst) {
    const int r = __builtin_amdgcn_readfirstlane(tile_row(t));  // (scalar buffer descriptors)
    copy.issue_rows(kbase + (size_t)r * D, N - r, kdst);
    copy.issue_rows(vbase + (size_t)r * D, N - r, vdst);
  };
  constexpr int DQ_COPIES = 2 * decltype(copy)::NI;
  if (T > 0) issue(0, lds, lds + 2 * TILE);

  bf16x8 qreg[DS], doreg[DS];
  float dlt = 0.f;  // Delta = rowsum(dO * O); each half-wave holds half of the row's features
#pragma unroll
  for (int s = 0; s < DS; ++s) {
    qreg[s] = qvalid ? *reinterpret_cast<const bf16x8*>(p.Q + qrow * D + 16 * s + 8 * g2) : zero_bf16x8();
    doreg[s] = qvalid ? *reinterpret_cast<const bf16x8*>(p.dO + qrow * D + 16 * s + 8 * g2) : zero_bf16x8();
    const bf16x8 o = qvalid ? *reinterpret_cast<const bf16x8*>(p.O + qrow * D + 16 * s + 8 * g2) : zero_bf16x8();
#pragma unroll
    for (int e = 0; e < 8; ++e) dlt += (float)doreg[s][e] * (float)o[e];
  }
  dlt = halves_sum(dlt);
  const float lse2 = qvalid ? p.LSE[qrow] * LOG2E : 0.f;
  if (qvalid && g2 == 0) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    const f32x2 v = {lse2, dlt};
    *reinterpret_cast<f32x2*>(p.rs + 2 * qrow) = v;
  }

  const LdsOperands<D> ops(lane);
  f32x16 dqacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) dqacc[db][e] = 0.f;

  wait_global_loads();
  __syncthreads();

  // The walk as in the forward kernel: first the key tiles FULL for the
  // whole query tile, in a loop with no visibility test, then the diagonal
  // ones, one 32-key block at a time, each wave skipping the blocks none of
  // its rows sees (wave-uniform windows; the per-row window is computed in
  // those steps only: this kernel has no registers to spare for caching it).
  const FullRange fr = full_range_vs_query_tile(qh, q0, q1, L, S, BM);
  const int wr0 = q0 + 32 * __builtin_amdgcn_readfirstlane(w), wr1 = imin(q1, wr0 + 32);
  const PosWindow uw_n = wave_keys_visible(qh, HALF_NOISY, wr0, wr1, L, S);
  const PosWindow uw_c = wave_keys_visible(qh, HALF_CLEAN, wr0, wr1, L, S);

  // One FULL key tile; restrict-qualified current and next buffers as in the
  // forward kernel, so the copy in flight does not make the compiler wait
  // before the reads of the current tile.  The copy of the next tile is
  // spread between the MFMAs (the last step copies its own tile again).
  auto tile_step = [&](const char* __restrict__ kcur, const char* __restrict__ vcur, char* __restrict__ knxt,
                       char* __restrict__ vnxt, int t) __attribute__((always_inline)) {
    {
      f32x16 sacc[KB], dpacc[KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          sacc[kb][e] = 0.f;
          dpacc[kb][e] = 0.f;
        }
      // the next tile's copy, one instruction per step of the loop below
      const int rn = __builtin_amdgcn_readfirstlane(tile_row(imin(t + 1, T - 1)));
      const __amdgpu_buffer_rsrc_t kn = make_buffer(kbase + (size_t)rn * D, (uint32_t)((N - rn) * D * 2));
      const __amdgpu_buffer_rsrc_t vn = make_buffer(vbase + (size_t)rn * D, (uint32_t)((N - rn) * D * 2));
      // S^T[key][q] = sum_d K[key][d] Q[q][d];  dP^T[key][q] = sum_d V[key][d] dO[q][d]
#pragma unroll
      for (int s = 0; s < DS; ++s) {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          sacc[kb] = mfma32(lds_rows<D>(kcur, ops.row_rel, s, kb), qreg[s], sacc[kb]);
          dpacc[kb] = mfma32(lds_rows<D>(vcur, ops.row_rel, s, kb), doreg[s], dpacc[kb]);
        }
        constexpr int NI = decltype(copy)::NI, PER = (2 * NI + DS - 1) / DS;  // copy instructions per step
#pragma unroll
        for (int x = 0; x < PER; ++x) {
          const int u = s * PER + x;
          if (u < NI) copy.issue_one(kn, knxt, u);
          else if (u < 2 * NI) copy.issue_one(vn, vnxt, u - NI);
        }
      }
      // operand reads four MFMAs ahead (a read's latency exceeds one MFMA),
      // the copy spread between the MFMAs
      pipeline_reads_and_copies<2 * DS * KB, 4, 1, DQ_COPIES>();
      // dS = P (dP - delta), every pair visible
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) sacc[kb][e] = fast_exp2(sacc[kb][e] * p.c - lse2) * (dpacc[kb][e] - dlt);
      bf16x8 dsb[PC];
#pragma unroll
      for (int c = 0; c < PC; ++c) dsb[c] = pack8(sacc[c >> 1], 8 * (c & 1));
      // dQ^T[d][q] += sum_key K^T[d][key] dS^T[key][q]
#pragma unroll
      for (int c = 0; c < PC; ++c)
#pragma unroll
        for (int db = 0; db < DB; ++db) dqacc[db] = mfma32(lds_tr<D>(kcur, ops.tr_rel0, ops.tr_rel1, c, db), dsb[c], dqacc[db]);
      // K^T operand reads four MFMAs ahead
      pipeline_lds_reads<PC * DB, 4, 2>();
    }
  };
  // One 32-key block kb of a diagonal key tile (the next tile's copy is
  // issued by the caller).
  auto block_step = [&](const char* __restrict__ kcur, const char* __restrict__ vcur, int kh, int k0, int kb)
                        __attribute__((always_inline)) {
    f32x16 sa, dpa;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      sa[e] = 0.f;
      dpa[e] = 0.f;
    }
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      sa = mfma32(lds_rows<D>(kcur, ops.row_rel, s, kb), qreg[s], sa);
      dpa = mfma32(lds_rows<D>(vcur, ops.row_rel, s, kb), doreg[s], dpa);
    }
    pipeline_lds_reads<2 * DS, 4, 1>();
    // dS = P (dP - delta) on the visible pairs, 0 elsewhere
    const PosWindow win = keys_visible_from(qh, kh, qblock0, L, S, qvalid);
    const unsigned span = (unsigned)(win.hi - win.lo);
    const int rel = k0 + 32 * kb + 4 * g2 - win.lo;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int e = 4 * i + jj;
        float pv = fast_exp2(sa[e] * p.c - lse2);
        pv = (unsigned)(rel + 8 * i + jj) < span ? pv : 0.f;
        sa[e] = pv * (dpa[e] - dlt);
      }
    const bf16x8 d0 = pack8(sa, 0), d1 = pack8(sa, 8);
#pragma unroll
    for (int db = 0; db < DB; ++db) dqacc[db] = mfma32(lds_tr<D>(kcur, ops.tr_rel0, ops.tr_rel1, 2 * kb, db), d0, dqacc[db]);
#pragma unroll
    for (int db = 0; db < DB; ++db)
      dqacc[db] = mfma32(lds_tr<D>(kcur, ops.tr_rel0, ops.tr_rel1, 2 * kb + 1, db), d1, dqacc[db]);
  };
  auto end_step = [&]() __attribute__((always_inline)) {
    compute_fence();
    wait_global_loads();
    __syncthreads();
  };
  const int t_main = __builtin_amdgcn_readfirstlane(imin(T, fr.full_prefix(BN)));
  for (int t = 0; t < t_main; ++t) {
    char* cur = lds + (t & 1) * TILE;
    char* nxt = lds + ((t + 1) & 1) * TILE;
    tile_step(cur, cur + 2 * TILE, nxt, nxt + 2 * TILE, t);
    end_step();
  }
  for (int t = t_main; t < T; ++t) {
    char* cur = lds + (t & 1) * TILE;
    char* nxt = lds + ((t + 1) & 1) * TILE;
    int kh, j;
    kl.at(t, kh, j);
    const int k0 = j * BN;
    const PosWindow uw = kh == HALF_NOISY ? uw_n : uw_c;
    issue(imin(t + 1, T - 1), nxt, nxt + 2 * TILE);
#pragma unroll 1
    for (int kb = 0; kb < KB; ++kb)  // (not unrolled: one block body in the loop)
      if (k0 + 32 * kb < uw.hi && k0 + 32 * kb + 32 > uw.lo) block_step(cur, cur + 2 * TILE, kh, k0, kb);
    end_step();
  }

  if (qvalid) {
    bf16* dqp = p.dQ + qrow * D + 4 * g2;
    const float sc = p.scale;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        st_bf16x4(dqp + db * 32 + 8 * i, dqacc[db][4 * i] * sc, dqacc[db][4 * i + 1] * sc,
                  dqacc[db][4 * i + 2] * sc, dqacc[db][4 * i + 3] * sc);
  }
}

template <int D>
hipError_t launch_dkdv_d(const Shape& s, const void* Q, const void* K, const void* V, const void* dO,
                         const float* rs, void* dK, void* dV, float* part, int* pair, hipStream_t st,
                         LaunchEvents ev) {
  DkvParams p;
  p.Q = static_cast<const bf16*>(Q);
  p.K = static_cast<const bf16*>(K);
  p.V = static_cast<const bf16*>(V);
  p.dO = static_cast<const bf16*>(dO);
  p.rs = rs;
  p.dK = static_cast<bf16*>(dK);
  p.dV = static_cast<bf16*>(dV);
  p.part = part;
  p.pair = pair;
  p.seq = s.seq;
  p.tile_slots = dkdv_tile_slots(s);
  p.L = s.L;
  p.S = s.S;
  p.Hq = s.Hq;
  p.Hkv = s.Hkv;
  p.G = s.G;
  p.nKT = cdiv(s.L, DKV_BN);
  p.nkv = s.B * s.Hkv;
  p.c = s.scale * LOG2E;
  p.scale = s.scale;
  // each clean key tile's walk in 2 or 4 parts, then the noisy key tiles
  // (packed sequences: grid sized by a bound on the key tiles of all sequences)
  const int rows = s.seq.cu ? packed_rows_bound(s.seq.T, s.B, s.L, DKV_BN) : p.nKT * s.B;
  if (dkdv_nsplit(s) == 4) {
    hipExtLaunchKernelGGL((dkdv_kernel<D, 4>), dim3(5 * rows * s.Hkv), dim3(512), 0, st, ev.start, ev.stop, 0, p);
  } else {
    hipExtLaunchKernelGGL((dkdv_kernel<D, 2>), dim3(3 * rows * s.Hkv), dim3(512), 0, st, ev.start, ev.stop, 0, p);
  }
  return hipGetLastError();
}

template <int D>
hipError_t launch_dq_d(const Shape& s, const void* Q, const void* K, const void* V, const void* dO, const void* O,
                       const float* LSE, float* rs, int* pair, void* dQ, hipStream_t st, LaunchEvents ev) {
  DqParams p;
  p.Q = static_cast<const bf16*>(Q);
  p.K = static_cast<const bf16*>(K);
  p.V = static_cast<const bf16*>(V);
  p.dO = static_cast<const bf16*>(dO);
  p.O = static_cast<const bf16*>(O);
  p.LSE = LSE;
  p.rs = rs;
  p.pair = pair;
  p.npair = (int)dkdv_pair_ints(s.B, s.Hkv, s.L);
  p.seq = s.seq;
  p.dQ = static_cast<bf16*>(dQ);
  p.L = s.L;
  p.S = s.S;
  p.Hq = s.Hq;
  p.Hkv = s.Hkv;
  p.G = s.G;
  p.nQT = cdiv(s.L, DQ_BM);
  p.nbh = s.B * s.Hq;
  p.c = s.scale * LOG2E;
  p.scale = s.scale;
  const dim3 grid(2 * p.nQT * p.nbh);
  hipExtLaunchKernelGGL(dq_kernel<D>, grid, dim3(256), 0, st, ev.start, ev.stop, 0, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bwd_dkdv(const Shape& s, const void* Q, const void* K, const void* V, const void* dO,
                           const float* rs, void* dK, void* dV, float* part, int* pair, hipStream_t st,
                           LaunchEvents ev) {
  if (s.D == 128) return launch_dkdv_d<128>(s, Q, K, V, dO, rs, dK, dV, part, pair, st, ev);
  return launch_dkdv_d<64>(s, Q, K, V, dO, rs, dK, dV, part, pair, st, ev);
}

hipError_t launch_bwd_dq(const Shape& s, const void* Q, const void* K, const void* V, const void* dO, const void* O,
                         const float* LSE, float* rs, int* pair, void* dQ, hipStream_t st, LaunchEvents ev) {
  if (s.D == 128) return launch_dq_d<128>(s, Q, K, V, dO, O, LSE, rs, pair, dQ, st, ev);
  return launch_dq_d<64>(s, Q, K, V, dO, O, LSE, rs, pair, dQ, st, ev);
}

}  // namespace bd
