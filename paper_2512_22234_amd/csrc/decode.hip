// Block-diffusion decoding over a KV cache for gfx950: the KV-cache reading
// of DiRL Section 2.1 used in rollouts.  While block k is denoised, its S noisy
// queries attend to the clean tokens of the blocks before it (the cache) and
// to each other in both directions (Eq. 2); nothing else exists yet, so there
// is no mask beyond the lengths.  Every cached K/V row is read once per
// (sequence, KV head, query tile) and serves up to 32 query rows of that KV
// head: the work is bound by HBM bandwidth, not by the MFMAs.
//
// Work items are (sequence b, KV head, 32-row tile of the G*S query rows);
// an item's keys are its cache_lens[b] cached rows followed by the block's S
// rows, cut into 32-key tiles (cache tiles, then block tiles; none straddles
// the two arrays).  Lay the tiles of all items end to end, in item order: T
// tiles in all.  Wave gw of the DEC_WAVES waves takes the contiguous run
// [gw*T/DEC_WAVES, (gw+1)*T/DEC_WAVES), whatever the lengths, so every wave
// streams the same number of bytes and a long cache is spread over many waves
// while short ones share a wave.  The lengths live on the device: every
// workgroup scans them once to find where its waves start.
//
// A wave keeps an online-softmax state for the item it is in and flushes it
// when the item or the run ends: an item that lies wholly inside one run is
// written out (O, LSE) at once; otherwise each run leaves its unnormalised O,
// max and sum in a partial slot, and dec_combine_kernel merges the runs of the
// item.  Slot gw + item is unique: two runs (gw, item) and (gw', item') with
// gw < gw' and item > item' cannot both hold tiles, since both the runs and
// the items are contiguous and in the same order.
//
// The waves never wait for each other: each double-buffers its own LDS tiles
// (copies go straight from HBM to LDS) and waits only for its own copies.
// Per tile: S^T = K Q^T (a lane owns a query column, as in the forward pass),
// P = exp2(c S - m) against a lazily moved reference max, O^T += V^T P^T with
// V^T read through the transposing LDS read.
#include "device.hpp"
#include "kernels.hpp"

namespace bd {
namespace {

struct DecParams {
  const bf16* Q;   // [B][Hq][S][D]
  const bf16* Kc;  // [B][Hkv][C][D]
  const bf16* Vc;
  const bf16* Kn;  // [B][Hkv][S][D]
  const bf16* Vn;
  const int* cache_lens;  // [B], device
  bf16* O;                // [B][Hq][S][D]
  float* LSE;             // [B][Hq][S]
  int4* desc;             // [item]: first run, last run (-1: the item was written directly), T
  float* part;            // [slot][32 rows][D + 4]: unnormalised O, max (log2 units), sum
  int B, S, Hq, Hkv, G, C, nqt;
  float c;  // scale * log2(e)
};

// Cache length of sequence b, clamped to [0, C].  `lens` is p.cache_lens
// passed as a restrict kernel argument: the compiler may then read it through
// the scalar cache where the index is uniform.
__device__ inline int dec_len(const DecParams& p, const int* __restrict__ lens, int b) {
  return imin(imax(lens[b], 0), p.C);
}
// Key tiles of an item of a sequence with cache length len.
__device__ inline int dec_tiles(const DecParams& p, int len) { return cdiv(len, DEC_KT) + cdiv(p.S, DEC_KT); }
// First tile of run gw (the runs cut T tiles into DEC_WAVES near-equal pieces).
__device__ inline int dec_run_start(int gw, int T) { return (int)(((long long)gw * T) / DEC_WAVES); }

// Position of a tile: sequence b (cache length len, nt tiles per item), item
// r of the sequence (KV head r / nqt, query tile r % nqt), tile j of the item.
struct DecPos {
  int b, len, nt, r, j;
};

template <int D>
struct DecSmem {
  static constexpr uint32_t TILE = DEC_KT * D * 2;  // bytes of one swizzled 32-key tile
  alignas(256) char buf[4][4 * TILE];                // per wave: K and V, double-buffered
  int wsum[4];                                       // prologue: per-wave sums of the scan
  int start_b[4], start_off[4];                      // where each wave's run starts
};

// The reference maximum of a row moves only when the row's scores exceed it
// by more than this (log2 units): P stays below 2^8, well inside bf16 and the
// float32 sums, and most tiles skip the rescale.
constexpr float DEC_SLACK = 8.0f;

template <int D>
__global__ __launch_bounds__(256, 1) void dec_kernel(DecParams p, const int* __restrict__ lens) {
  constexpr int DS = D / 16, DB = D / 32, PST = D + 4;
  using Smem = DecSmem<D>;
  __shared__ Smem sm;

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, g2 = lane >> 5;
  const int I = p.Hkv * p.nqt;  // items per sequence

  // ---- prologue: T, and the position of each wave's first tile ----
  // thread t sums the tiles per item of sequences [t*cpt, (t+1)*cpt)
  const int cpt = cdiv(p.B, 256);
  const int c0 = imin(p.B, tid * cpt), c1 = imin(p.B, c0 + cpt);
  int csum = 0;
#pragma unroll 4
  for (int b = c0; b < c1; ++b) csum += dec_tiles(p, dec_len(p, lens, b));
  int incl = csum;  // inclusive scan over the wave
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(incl, o, 64);
    if (lane >= o) incl += u;
  }
  if (lane == 63) sm.wsum[w] = incl;
  __syncthreads();
  int before = 0, total = 0;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int s = sm.wsum[v];
    before += v < w ? s : 0;
    total += s;
  }
  const int excl = before + incl - csum;  // tiles per item of the sequences before c0
  const int T = total * I;                // checked on the host to fit in 31 bits
  // the thread whose sequences hold a wave's first tile records where it lies
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int x0 = dec_run_start(blockIdx.x * 4 + v, T);
    if (csum > 0 && excl * I <= x0 && x0 < (excl + csum) * I) {
      int pb = excl;
      for (int b = c0; b < c1; ++b) {
        const int nt = dec_tiles(p, dec_len(p, lens, b));
        if (x0 < (pb + nt) * I) {
          sm.start_b[v] = b;
          sm.start_off[v] = x0 - pb * I;
          break;
        }
        pb += nt;
      }
    }
  }
  __syncthreads();

  // ---- this wave's run ----
  const int gw = blockIdx.x * 4 + w;
  const int x0 = dec_run_start(gw, T), x1 = dec_run_start(gw + 1, T);
  if (x0 >= x1) return;
  DecPos pc;
  pc.b = __builtin_amdgcn_readfirstlane(sm.start_b[w]);
  const int off = __builtin_amdgcn_readfirstlane(sm.start_off[w]);
  pc.len = __builtin_amdgcn_readfirstlane(dec_len(p, lens, pc.b));
  pc.nt = dec_tiles(p, pc.len);
  pc.r = off / pc.nt;
  pc.j = off - pc.r * pc.nt;
  const int S = p.S;

  auto advance = [&](DecPos q) {
    if (++q.j == q.nt) {
      q.j = 0;
      if (++q.r == I) {
        q.r = 0;
        if (++q.b < p.B) {
          q.len = __builtin_amdgcn_readfirstlane(dec_len(p, lens, q.b));
          q.nt = dec_tiles(p, q.len);
        }
      }
    }
    return q;
  };
  // this lane's query row of item (b, r): row qt*32 + l32 of the G*S rows of
  // KV head r / nqt (those rows are consecutive in Q, O and LSE).  A lane
  // past the last row takes the last row instead: its score column is
  // computed like the others (columns never mix) and never stored.
  auto query_row = [&](DecPos q, bool& valid) {
    const int hkv = q.r / p.nqt, R = (q.r - hkv * p.nqt) * DEC_QT + l32;
    valid = R < p.G * S;
    return ((size_t)q.b * p.Hq + (size_t)hkv * p.G) * S + (valid ? R : p.G * S - 1);
  };
  struct QRows {
    bf16x8 v[DS];
  };
  auto load_q = [&](DecPos q) {
    bool valid;
    const size_t row = query_row(q, valid);
    QRows r;
#pragma unroll
    for (int s = 0; s < DS; ++s) r.v[s] = *reinterpret_cast<const bf16x8*>(p.Q + row * D + 16 * s + 8 * g2);
    return r;
  };

  const TileCopy<D, DEC_KT, 64> copy(lane);  // one wave copies a whole tile
  constexpr int NI = decltype(copy)::NI;
  // copy K and V of the tile at q to dst, dst + TILE
  auto issue = [&](DecPos q, char* dst) {
    const size_t grp = (size_t)q.b * p.Hkv + q.r / p.nqt;
    const int ntc = cdiv(q.len, DEC_KT);
    const bool cached = q.j < ntc;
    const int r0 = (cached ? q.j : q.j - ntc) * DEC_KT;
    const int left = (cached ? q.len : S) - r0;
    const size_t off2 = (cached ? grp * p.C : grp * S) * D + (size_t)r0 * D;
    copy.issue_rows((cached ? p.Kc : p.Kn) + off2, left, dst);
    copy.issue_rows((cached ? p.Vc : p.Vn) + off2, left, dst + Smem::TILE);
  };

  const LdsOperands<D> ops(lane);
  QRows qreg, qnext;
  f32x16 oacc[DB];
  float m, lsum;
  auto reset = [&]() {
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int e = 0; e < 16; ++e) oacc[db][e] = 0.f;
    m = -INFINITY;
    lsum = 0.f;
  };
  reset();
  char* const mine = sm.buf[w];
  qreg = load_q(pc);
  issue(pc, mine);
  int item_start = x0 - pc.j;  // flat index of the current item's first tile
  int seg_j0 = pc.j;           // tile of the item this run's segment starts at

  // Write out the state of the current item's segment, which ends at tile pc.j.
  auto flush = [&]() {
    const int item = pc.b * I + pc.r;
    const bool ends = pc.j == pc.nt - 1;
    bool valid;
    const size_t qrow = query_row(pc, valid);
    const float Lrow = halves_sum(lsum);
    if (seg_j0 == 0 && ends) {
      if (valid) {
        const float inv = 1.f / Lrow;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          bf16* op = p.O + qrow * D + 32 * db + 4 * g2;
#pragma unroll
          for (int i = 0; i < 4; ++i)
            st_bf16x4(op + 8 * i, oacc[db][4 * i] * inv, oacc[db][4 * i + 1] * inv, oacc[db][4 * i + 2] * inv,
                      oacc[db][4 * i + 3] * inv);
        }
        if (g2 == 0) p.LSE[qrow] = (m + __log2f(Lrow)) * LN2;
      }
      if (lane == 0) p.desc[item] = int4{0, -1, T, 0};
      return;
    }
    if (valid) {
      float* pr = p.part + ((size_t)(gw + item) * DEC_QT + l32) * PST;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const f32x4 v = {oacc[db][4 * i], oacc[db][4 * i + 1], oacc[db][4 * i + 2], oacc[db][4 * i + 3]};
          *reinterpret_cast<f32x4*>(pr + 32 * db + 8 * i + 4 * g2) = v;
        }
      if (g2 == 0) *reinterpret_cast<f32x4*>(pr + D) = f32x4{m, Lrow, 0.f, 0.f};
    }
    if (ends && lane == 0) {
      // the runs holding this item: from the one holding its first tile to this one
      const int first = (int)((((long long)item_start + 1) * DEC_WAVES - 1) / T);
      p.desc[item] = int4{first, gw, T, 0};
    }
  };

  // One tile: `cur` holds the tile at pc; the copy of the next tile (at pn,
  // if this run has one) goes to `nxt`.  The restrict qualifiers tell the
  // compiler that the copy in flight does not touch `cur`, so its reads need
  // not wait for it.  Query rows of the next item are loaded a tile ahead,
  // after the wait for the current tile (which covers the current item's
  // query rows, loaded before the next tile's copy): copies and query loads
  // complete in issue order.
  auto step = [&](const char* __restrict__ cur, char* __restrict__ nxt, DecPos pn, bool more,
                  bool new_item) __attribute__((always_inline)) {
    compute_fence();  // the reads of the buffer about to be refilled are done
    // (the query-row copy sits in both branches so that the compiler's own
    // wait for it counts the copy just issued on the first one)
    if (more) {
      issue(pn, nxt);
      wait_global_loads_but<2 * NI>();  // the tile at pc has landed (this wave's own copy)
      if (new_item) qreg = qnext;
      if (pn.j == 0) qnext = load_q(pn);
    } else {
      wait_global_loads();
      if (new_item) qreg = qnext;
    }
    const int ntc = cdiv(pc.len, DEC_KT);
    const int nvalid = pc.j < ntc ? pc.len - pc.j * DEC_KT : S - (pc.j - ntc) * DEC_KT;  // keys that exist

    // S^T[key][query] = sum_d K[key][d] Q[query][d]
    f32x16 sacc;
#pragma unroll
    for (int e = 0; e < 16; ++e) sacc[e] = 0.f;
#pragma unroll
    for (int s = 0; s < DS; ++s) sacc = mfma32(lds_rows<D>(cur, ops.row_rel, s, 0), qreg.v[s], sacc);
    if (nvalid < DEC_KT) {
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          if (8 * i4 + 4 * g2 + jj >= nvalid) sacc[4 * i4 + jj] = -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sacc[e]);
    mx = halves_max(mx) * p.c;
    const bool grow = mx > m + DEC_SLACK;
    if (__any(grow)) {
      const float alpha = grow ? fast_exp2(m - mx) : 1.f;
      m = grow ? mx : m;
      lsum *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[db][e] *= alpha;
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float x = fast_exp2(sacc[e] * p.c - m);
      sacc[e] = x;
      lsum += x;
    }
    const bf16x8 pb[2] = {pack8(sacc, 0), pack8(sacc, 8)};
    // O^T[d][query] += sum_key V^T[d][key] P^T[key][query]
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int db = 0; db < DB; ++db)
        oacc[db] = mfma32(lds_tr<D>(cur + Smem::TILE, ops.tr_rel0, ops.tr_rel1, c, db), pb[c], oacc[db]);
  };

  for (int x = x0, i = 0; x < x1; ++x, ++i) {
    const DecPos pn = advance(pc);
    const bool more = x + 1 < x1;
    step(mine + (i & 1) * 2 * Smem::TILE, mine + ((i + 1) & 1) * 2 * Smem::TILE, pn, more, x > x0 && pc.j == 0);
    if (!more || pn.j == 0) {
      flush();
      if (more) {  // the next tile starts the next item
        reset();
        item_start += pc.nt;
        seg_j0 = 0;
      }
    }
    pc = pn;
  }
}

// Merge the runs of each query row of an item held by several waves:
// O = sum_r 2^(m_r - M) O_r / sum_r 2^(m_r - M) l_r with M = max_r m_r, over
// the runs of waves first..last that hold tiles, merged in one pass (the
// running maximum moves as runs are added, so every run's loads are
// independent of the others' results).  One thread per (query row, 4
// features); rows are those of Q, so no thread is spent on padding rows of a
// query tile.
template <int D>
__global__ __launch_bounds__(256) void dec_combine_kernel(DecParams p) {
  constexpr int TPR = D / 4, PST = D + 4;
  const size_t gid = (size_t)blockIdx.x * 256 + threadIdx.x;
  const size_t qrow = gid / TPR;  // row of Q: ((b * Hq + h) * S + s)
  const int q4 = (int)(gid % TPR);
  const int GS = p.G * p.S;
  if (qrow >= (size_t)p.B * p.Hkv * GS) return;
  const int R = (int)(qrow % GS);
  const size_t bh = qrow / GS;  // b * Hkv + hkv
  const int item = (int)(bh * p.nqt) + R / DEC_QT, r = R % DEC_QT;
  const int4 d = p.desc[item];
  if (d.y < 0) return;  // written by the decode kernel itself
  const int T = d.z;
  float M = -INFINITY, Lr = 0.f;
  f32x4 o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int gw = d.x; gw <= d.y; ++gw) {
    const float* ps = p.part + ((size_t)(gw + item) * DEC_QT + r) * PST;
    const f32x4 ml = *reinterpret_cast<const f32x4*>(ps + D);
    const f32x4 v = *reinterpret_cast<const f32x4*>(ps + 4 * q4);
    if (dec_run_start(gw, T) == dec_run_start(gw + 1, T)) continue;  // a wave without tiles wrote nothing
    const float Mn = fmaxf(M, ml[0]);
    const float a = fast_exp2(M - Mn), c = fast_exp2(ml[0] - Mn);  // a = 0 for the first run (M = -inf)
    Lr = Lr * a + ml[1] * c;
    o = o * a + v * c;
    M = Mn;
  }
  const float inv = 1.f / Lr;
  st_bf16x4(p.O + qrow * D + 4 * q4, o[0] * inv, o[1] * inv, o[2] * inv, o[3] * inv);
  if (q4 == 0) p.LSE[qrow] = (M + __log2f(Lr)) * LN2;
}

template <int D>
hipError_t launch_decode_d(const DecodeShape& s, const void* Q, const void* Kc, const void* Vc, const void* Kn,
                           const void* Vn, const int* cache_lens, void* O, float* LSE, void* ws, hipStream_t st) {
  DecParams p;
  p.Q = static_cast<const bf16*>(Q);
  p.Kc = static_cast<const bf16*>(Kc);
  p.Vc = static_cast<const bf16*>(Vc);
  p.Kn = static_cast<const bf16*>(Kn);
  p.Vn = static_cast<const bf16*>(Vn);
  p.cache_lens = cache_lens;
  p.O = static_cast<bf16*>(O);
  p.LSE = LSE;
  p.desc = static_cast<int4*>(ws);
  p.part = reinterpret_cast<float*>(static_cast<char*>(ws) + decode_desc_bytes(s));
  p.B = s.B;
  p.S = s.S;
  p.Hq = s.Hq;
  p.Hkv = s.Hkv;
  p.G = s.Hq / s.Hkv;
  p.C = s.C;
  p.nqt = decode_query_tiles(s);
  p.c = s.scale * LOG2E;
  hipLaunchKernelGGL(dec_kernel<D>, dim3(DEC_WAVES / 4), dim3(256), 0, st, p, cache_lens);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t threads = (size_t)s.B * s.Hq * s.S * (D / 4);
  hipLaunchKernelGGL(dec_combine_kernel<D>, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const DecodeShape& s, const void* Q, const void* Kc, const void* Vc, const void* Kn,
                         const void* Vn, const int* cache_lens, void* O, float* LSE, void* ws, hipStream_t st) {
  if (s.D == 128) return launch_decode_d<128>(s, Q, Kc, Vc, Kn, Vn, cache_lens, O, LSE, ws, st);
  return launch_decode_d<64>(s, Q, Kc, Vc, Kn, Vn, cache_lens, O, LSE, ws, st);
}

}  // namespace bd
