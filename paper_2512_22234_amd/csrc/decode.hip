// Block-diffusion decoding over a KV cache for gfx950: the KV-cache reading
// of DiRL Section 2.1 used in rollouts.  While block k is denoised, its S noisy
// queries attend to the clean tokens of the blocks before it (the cache) and
// to each other in both directions (Eq. 2); nothing else exists yet, so there
// is no mask beyond the lengths.  Every cached K/V row is read once per
// (sequence, KV head) and serves all G*S query rows of that KV head: the work
// is bound by HBM bandwidth, not by the MFMAs.
//
// Work item: (sequence b, KV head, 32-row tile of the G*S query rows).  The
// keys of a sequence are its cache_lens[b] cached rows followed by the
// block's S noisy rows, cut into 32-key tiles (cache tiles, then block tiles;
// none straddles the two arrays), and split into runs of `tps` tiles, one
// workgroup per (item, split).  The four waves of a workgroup take alternate
// tiles of the run, each double-buffering its own LDS tiles (so the loop needs
// no workgroup barrier), and merge their online-softmax states through LDS at
// the end.  An item whose keys fit one split writes O and LSE at once; the
// splits of a longer one leave (unnormalised O, max, sum) per row and
// dec_combine_kernel merges them.
//
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
  float* part;            // [item][split][32 rows][D + 4]: unnormalised O, max (log2 units), sum
  int S, Hq, Hkv, G, C, max_len, nqt, nsplit, tps;
  float c;  // scale * log2(e)
};

// Cache length of sequence b, clamped to the cache and to the launch's bound.
__device__ inline int dec_len(const DecParams& p, int b) {
  return imin(imax(__builtin_amdgcn_readfirstlane(p.cache_lens[b]), 0), imin(p.C, p.max_len));
}

template <int D>
struct DecSmem {
  static constexpr uint32_t TILE = DEC_KT * D * 2;  // bytes of one swizzled 32-key tile
  static constexpr uint32_t WAVE = 4 * TILE;         // per wave: K and V, double-buffered
  static_assert(WAVE >= (64 * 16 * (D / 32) + 2 * 64) * 4, "the merge reuses a wave's tiles");
  alignas(256) char buf[4][WAVE];
};

// The reference maximum of a row moves only when the row's scores exceed it
// by more than this (log2 units): P stays below 2^8, well inside bf16 and the
// float32 sums, and most tiles skip the rescale.
constexpr float DEC_SLACK = 8.0f;

template <int D>
__global__ __launch_bounds__(256, 1) void dec_kernel(DecParams p) {
  constexpr int DS = D / 16, DB = D / 32, PST = D + 4;
  using Smem = DecSmem<D>;
  __shared__ Smem sm;

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, g2 = lane >> 5;

  // id = ((b * Hkv + hkv) * nqt + qt) * nsplit + sp
  const int id = blockIdx.x;
  const int sp = id % p.nsplit;
  const int item = id / p.nsplit;
  const int qt = item % p.nqt;
  const int grp = item / p.nqt;  // b * Hkv + hkv
  const int b = grp / p.Hkv, hkv = grp - b * p.Hkv;
  const int S = p.S;
  const int len = dec_len(p, b);
  const int ntc = cdiv(len, DEC_KT), nt = ntc + cdiv(S, DEC_KT);
  const int ns = cdiv(nt, p.tps);  // splits this item uses
  if (sp >= ns) return;
  const int t0 = sp * p.tps, t1 = imin(nt, t0 + p.tps);

  // this lane's query row R of the G*S rows of the KV head (head hkv*G + R/S,
  // block row R%S): those rows are consecutive in Q, O and LSE
  const int R = qt * DEC_QT + l32;
  const bool qvalid = R < p.G * S;
  const size_t qrow = ((size_t)b * p.Hq + (size_t)hkv * p.G) * S + (qvalid ? R : 0);

  bf16x8 qreg[DS];
#pragma unroll
  for (int s = 0; s < DS; ++s)
    qreg[s] = qvalid ? *reinterpret_cast<const bf16x8*>(p.Q + qrow * D + 16 * s + 8 * g2) : zero_bf16x8();

  const LdsOperands<D> ops(lane);
  const TileCopy<D, DEC_KT, 64> copy(lane);  // one wave copies a whole tile
  constexpr int NI = decltype(copy)::NI;
  const size_t kvc = (size_t)grp * p.C * D, kvn = (size_t)grp * S * D;
  // copy K and V of key tile t (cache tiles, then block tiles) to dst, dst + TILE
  auto issue = [&](int t, char* dst) {
    const bool cached = t < ntc;
    const int r0 = (cached ? t : t - ntc) * DEC_KT;
    const int left = (cached ? len : S) - r0;
    const size_t off = (cached ? kvc : kvn) + (size_t)r0 * D;
    copy.issue_rows((cached ? p.Kc : p.Kn) + off, left, dst);
    copy.issue_rows((cached ? p.Vc : p.Vn) + off, left, dst + Smem::TILE);
  };

  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[db][e] = 0.f;
  float m = -INFINITY, lsum = 0.f;

  char* const mine = sm.buf[w];
  const int nloc = t1 - t0 > w ? (t1 - t0 - w + 3) / 4 : 0;  // this wave's tiles t0 + w + 4i
  if (nloc > 0) issue(t0 + w, mine);
  // One tile: `cur` holds tile t; the copy of the wave's next tile (if any)
  // goes to `nxt`.  The restrict qualifiers tell the compiler that the copy
  // in flight does not touch `cur`, so its reads need not wait for it.
  auto step = [&](const char* __restrict__ cur, char* __restrict__ nxt, int t, bool more)
                  __attribute__((always_inline)) {
    compute_fence();  // the reads of the buffer about to be refilled are done
    if (more) {
      issue(t + 4, nxt);
      wait_global_loads_but<2 * NI>();  // tile t has landed (this wave's own copy: no barrier needed)
    } else {
      wait_global_loads();
    }
    const int nvalid = t < ntc ? len - t * DEC_KT : S - (t - ntc) * DEC_KT;  // keys of this tile that exist

    // S^T[key][query] = sum_d K[key][d] Q[query][d]
    f32x16 sacc;
#pragma unroll
    for (int e = 0; e < 16; ++e) sacc[e] = 0.f;
#pragma unroll
    for (int s = 0; s < DS; ++s) sacc = mfma32(lds_rows<D>(cur, ops.row_rel, s, 0), qreg[s], sacc);
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
  for (int i = 0; i < nloc; ++i) {
    char* cur = mine + (i & 1) * 2 * Smem::TILE;
    char* nxt = mine + ((i + 1) & 1) * 2 * Smem::TILE;
    step(cur, nxt, t0 + w + 4 * i, i + 1 < nloc);
  }

  // Merge the four waves' states: each wave leaves its O^T (16 values per
  // feature block per lane), reference max and per-lane sum in its own tiles
  // (no copy into them is in flight any more); wave w then merges feature
  // block w for every row.
  float* st = reinterpret_cast<float*>(mine);
  compute_fence();
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) st[(db * 16 + e) * 64 + lane] = oacc[db][e];
  st[DB * 16 * 64 + lane] = m;
  st[DB * 16 * 64 + 64 + lane] = lsum;
  __syncthreads();
  if (w >= DB || !qvalid) return;
  float mw[4], M = -INFINITY;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    mw[v] = reinterpret_cast<const float*>(sm.buf[v])[DB * 16 * 64 + lane];
    M = fmaxf(M, mw[v]);
  }
  float Lrow = 0.f;
  float o[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) o[e] = 0.f;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const float* sv = reinterpret_cast<const float*>(sm.buf[v]);
    const float a = mw[v] == -INFINITY ? 0.f : fast_exp2(mw[v] - M);  // a wave without tiles adds nothing
    Lrow += a * (sv[DB * 16 * 64 + 64 + lane] + sv[DB * 16 * 64 + 64 + (lane ^ 32)]);
#pragma unroll
    for (int e = 0; e < 16; ++e) o[e] += a * sv[(w * 16 + e) * 64 + lane];
  }
  // lane (l32, g2) holds features 32w + 8i + 4*g2 + j of its row at o[4i + j]
  if (ns == 1) {
    const float inv = 1.f / Lrow;
    bf16* op = p.O + qrow * D + 32 * w + 4 * g2;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      st_bf16x4(op + 8 * i, o[4 * i] * inv, o[4 * i + 1] * inv, o[4 * i + 2] * inv, o[4 * i + 3] * inv);
    if (w == 0 && g2 == 0) p.LSE[qrow] = (M + __log2f(Lrow)) * LN2;
  } else {
    float* pr = p.part + ((size_t)id * DEC_QT + l32) * PST;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const f32x4 v = {o[4 * i], o[4 * i + 1], o[4 * i + 2], o[4 * i + 3]};
      *reinterpret_cast<f32x4*>(pr + 32 * w + 8 * i + 4 * g2) = v;
    }
    if (w == 0 && g2 == 0) {
      pr[D] = M;
      pr[D + 1] = Lrow;
    }
  }
}

// Merge the splits of each query row of items that needed more than one:
// O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s with M = max_s m_s.
// One thread per (item, row, 4 features).
template <int D>
__global__ __launch_bounds__(256) void dec_combine_kernel(DecParams p, int nitems) {
  constexpr int TPR = D / 4, PST = D + 4;
  const size_t gid = (size_t)blockIdx.x * 256 + threadIdx.x;
  const size_t rowid = gid / TPR;  // item * 32 + r
  const int q4 = (int)(gid % TPR);
  if (rowid >= (size_t)nitems * DEC_QT) return;
  const int item = (int)(rowid / DEC_QT), r = (int)(rowid % DEC_QT);
  const int qt = item % p.nqt, grp = item / p.nqt;
  const int b = grp / p.Hkv, hkv = grp - b * p.Hkv;
  const int R = qt * DEC_QT + r;
  if (R >= p.G * p.S) return;
  const int len = dec_len(p, b);
  const int ns = cdiv(cdiv(len, DEC_KT) + cdiv(p.S, DEC_KT), p.tps);
  if (ns == 1) return;  // written by the decode kernel itself
  const size_t qrow = ((size_t)b * p.Hq + (size_t)hkv * p.G) * p.S + R;
  const float* base = p.part + ((size_t)item * p.nsplit * DEC_QT + r) * PST;
  const size_t sstride = (size_t)DEC_QT * PST;
  float M = -INFINITY;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, base[s * sstride + D]);
  float Lr = 0.f;
  f32x4 o = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < ns; ++s) {
    const float* ps = base + s * sstride;
    const float a = fast_exp2(ps[D] - M);  // every split of the item holds at least one key
    Lr += a * ps[D + 1];
    o += a * *reinterpret_cast<const f32x4*>(ps + 4 * q4);
  }
  const float inv = 1.f / Lr;
  st_bf16x4(p.O + qrow * D + 4 * q4, o[0] * inv, o[1] * inv, o[2] * inv, o[3] * inv);
  if (q4 == 0) p.LSE[qrow] = (M + __log2f(Lr)) * LN2;
}

template <int D>
hipError_t launch_decode_d(const DecodeShape& s, const void* Q, const void* Kc, const void* Vc, const void* Kn,
                           const void* Vn, const int* cache_lens, void* O, float* LSE, float* part, hipStream_t st) {
  DecParams p;
  p.Q = static_cast<const bf16*>(Q);
  p.Kc = static_cast<const bf16*>(Kc);
  p.Vc = static_cast<const bf16*>(Vc);
  p.Kn = static_cast<const bf16*>(Kn);
  p.Vn = static_cast<const bf16*>(Vn);
  p.cache_lens = cache_lens;
  p.O = static_cast<bf16*>(O);
  p.LSE = LSE;
  p.part = part;
  p.S = s.S;
  p.Hq = s.Hq;
  p.Hkv = s.Hkv;
  p.G = s.Hq / s.Hkv;
  p.C = s.C;
  p.max_len = s.max_len;
  p.nqt = decode_query_tiles(s);
  p.nsplit = decode_splits(s);
  p.tps = s.tps;
  p.c = s.scale * LOG2E;
  const int nitems = s.B * s.Hkv * p.nqt;
  hipLaunchKernelGGL(dec_kernel<D>, dim3((unsigned)nitems * p.nsplit), dim3(256), 0, st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.nsplit == 1) return e;
  const size_t threads = (size_t)nitems * DEC_QT * (D / 4);
  hipLaunchKernelGGL(dec_combine_kernel<D>, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st, p, nitems);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const DecodeShape& s, const void* Q, const void* Kc, const void* Vc, const void* Kn,
                         const void* Vn, const int* cache_lens, void* O, float* LSE, float* part, hipStream_t st) {
  if (s.D == 128) return launch_decode_d<128>(s, Q, Kc, Vc, Kn, Vn, cache_lens, O, LSE, part, st);
  return launch_decode_d<64>(s, Q, Kc, Vc, Kn, Vn, cache_lens, O, LSE, part, st);
}

}  // namespace bd
