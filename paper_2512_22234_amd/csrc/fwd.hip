// Forward pass of block-diffusion masked attention (DiRL Section 4.1, mask of
// Eq. 1 / Eq. 2) for gfx950.
//
// One workgroup = one (batch, query head, query tile of 128 rows); four waves,
// each owning 32 query rows.  Scores are computed transposed, S^T = K Q^T, so
// that each lane owns one query column: the row max needs one cross-lane
// exchange (lane l <-> l+32) per key tile and the running row sum stays a
// per-lane partial until the epilogue.  O^T = V^T P^T reuses the score
// accumulator directly as the bf16 B operand; its A operand V^T is read from
// the row-major V tile with the transposing LDS read (see device.hpp).
//
// Key tiles (64 keys) are visited in the order given by the exact tile
// classification: FULL tiles run with no per-element test, PARTIAL tiles
// apply the visibility rule per element, EMPTY tiles are never loaded.  K and
// V tiles are double-buffered in LDS; the next tile's global loads are in
// flight while the current one is computed.
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
  int L, S, Hq, Hkv, G, nQT, nbh;
  float c;  // scale * log2(e)
};

template <int D>
struct FwdSmem {
  static constexpr int BN = FWD_BN;
  static constexpr int KS = D + 8;  // K/V row stride (elements), 16-byte pad against bank conflicts
  bf16 k[2][BN * KS];
  bf16 v[2][BN * KS];
  alignas(16) int kblk[2][BN];
};

template <int D>
__global__ __launch_bounds__(256, 2) void fwd_kernel(FwdParams p) {
  constexpr int BM = FWD_BM, BN = FWD_BN;
  constexpr int DS = D / 16, DB = D / 32, KB = BN / 32, PC = BN / 16;
  constexpr int KS = FwdSmem<D>::KS;
  constexpr int NCH = BN * D / 8 / 256;  // 16-byte chunks per thread, for each of K and V
  static_assert(NCH * 256 * 8 == BN * D, "tile must split evenly over 256 threads");
  __shared__ FwdSmem<D> sm;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, g2 = lane >> 5;
  const int L = p.L, S = p.S, N = 2 * L;

  // Heaviest query tiles first (work grows with the tile index), noisy before
  // clean; heads remapped so a KV group stays on one XCD.
  const int id = blockIdx.x;
  const int rank = id / p.nbh;
  const int bh = xcd_head_remap(id - rank * p.nbh, p.nbh, p.G);
  const int qi = p.nQT - 1 - (rank >> 1);
  const int qh = rank & 1;
  const int b = bh / p.Hq, hq = bh - b * p.Hq, hk = hq / p.G;
  const int q0 = qi * BM, q1 = imin(L, q0 + BM);

  const size_t kvbase = (size_t)(b * p.Hkv + hk) * N * D;

  const int r = q0 + w * 32 + l32;  // this lane's query row (local to its half)
  const bool qvalid = r < q1;
  const int bq = qvalid ? r / S : QBLK_INVALID;
  const int prow = qh * L + r;

  bf16x8 qreg[DS];
  {
    const bf16* qp = p.Q + ((size_t)bh * N + prow) * D + 8 * g2;
#pragma unroll
    for (int s = 0; s < DS; ++s)
      qreg[s] = qvalid ? *reinterpret_cast<const bf16x8*>(qp + 16 * s) : zero_bf16x8();
  }

  const KeyTileList kl = key_tiles_for_query_tile(qh, qi, L, S, BM, BN);
  const int T = kl.count();

  u32x4 kst[NCH], vst[NCH];
  int kbst = 0;
  auto load_tile = [&](int t) {
    int kh, j;
    kl.at(t, kh, j);
    const bf16* kp = p.K + kvbase + (size_t)kh * L * D;
    const bf16* vp = p.V + kvbase + (size_t)kh * L * D;
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int c = tid + 256 * u;
      const int row = c / (D / 8), col8 = c % (D / 8);
      kst[u] = ld16_rows(kp, j * BN + row, L, D, col8 * 8);
      vst[u] = ld16_rows(vp, j * BN + row, L, D, col8 * 8);
    }
    if (tid < BN) {
      const int key = j * BN + tid;
      kbst = key < L ? key / S : KBLK_INVALID;
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int c = tid + 256 * u;
      const int row = c / (D / 8), col8 = c % (D / 8);
      st16(&sm.k[buf][row * KS + col8 * 8], kst[u]);
      st16(&sm.v[buf][row * KS + col8 * 8], vst[u]);
    }
    if (tid < BN) sm.kblk[buf][tid] = kbst;
  };

  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[db][e] = 0.f;
  float m = -INFINITY, lsum = 0.f;

  if (T > 0) {
    load_tile(0);
    store_tile(0);
  }
  wait_global_loads();  // Q rows are in registers; the loop only waits on its own prefetch
  __syncthreads();

  for (int t = 0; t < T; ++t) {
    const int buf = t & 1;
    if (t + 1 < T) load_tile(t + 1);
    int kh, j;
    kl.at(t, kh, j);
    const int k0 = j * BN, k1 = imin(L, k0 + BN);
    const int cls = classify_pair(qh, q0, q1, kh, k0, k1, S, (q1 - q0) == BM && (k1 - k0) == BN);
    if (cls != TILE_EMPTY) {
      f32x16 sacc[KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) sacc[kb][e] = 0.f;
      // S^T[key][query] = sum_d K[key][d] Q[query][d]
#pragma unroll
      for (int s = 0; s < DS; ++s)
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          const bf16x8 a = lds_bf16x8(&sm.k[buf][(kb * 32 + l32) * KS + 16 * s + 8 * g2]);
          sacc[kb] = mfma32(a, qreg[s], sacc[kb]);
        }
      if (cls == TILE_PARTIAL) {
        const BlockWindow win = key_window(qh, kh, bq);
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int4 kb4 = *reinterpret_cast<const int4*>(&sm.kblk[buf][kb * 32 + 8 * i + 4 * g2]);
            const int kbv[4] = {kb4.x, kb4.y, kb4.z, kb4.w};
#pragma unroll
            for (int jj = 0; jj < 4; ++jj)
              sacc[kb][4 * i + jj] = win.has(kbv[jj]) ? sacc[kb][4 * i + jj] : -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sacc[kb][e]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mnew = fmaxf(m, mx * p.c);
      const float muse = (mnew == -INFINITY) ? 0.f : mnew;
      const float alpha = fast_exp2(m - muse);
      m = mnew;
      float ps = 0.f;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float x = fast_exp2(sacc[kb][e] * p.c - muse);
          sacc[kb][e] = x;
          ps += x;
        }
      lsum = lsum * alpha + ps;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[db][e] *= alpha;
      bf16x8 pb[PC];
#pragma unroll
      for (int c = 0; c < PC; ++c) pb[c] = pack8(sacc[c >> 1], 8 * (c & 1));
      // O^T[d][query] += sum_key V^T[d][key] P^T[key][query]
#pragma unroll
      for (int c = 0; c < PC; ++c)
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const bf16x8 a = lds_read_tr(sm.v[buf], KS, 16 * c, db * 32, lane);
          oacc[db] = mfma32(a, pb[c], oacc[db]);
        }
    }
    compute_fence();
    if (t + 1 < T) store_tile(buf ^ 1);
    __syncthreads();
  }

  const float lt = lsum + __shfl_xor(lsum, 32);
  if (qvalid) {
    const float inv = 1.f / lt;
    bf16* op = p.O + ((size_t)bh * N + prow) * D + 4 * g2;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        st_bf16x4(op + db * 32 + 8 * i, oacc[db][4 * i] * inv, oacc[db][4 * i + 1] * inv,
                  oacc[db][4 * i + 2] * inv, oacc[db][4 * i + 3] * inv);
    if (g2 == 0) p.LSE[(size_t)bh * N + prow] = (m + log2f(lt)) * LN2;
  }
}

template <int D>
hipError_t launch_fwd_d(const Shape& s, const void* Q, const void* K, const void* V, void* O,
                        float* LSE, hipStream_t st) {
  FwdParams p;
  p.Q = static_cast<const bf16*>(Q);
  p.K = static_cast<const bf16*>(K);
  p.V = static_cast<const bf16*>(V);
  p.O = static_cast<bf16*>(O);
  p.LSE = LSE;
  p.L = s.L;
  p.S = s.S;
  p.Hq = s.Hq;
  p.Hkv = s.Hkv;
  p.G = s.G;
  p.nQT = cdiv(s.L, FWD_BM);
  p.nbh = s.B * s.Hq;
  p.c = s.scale * LOG2E;
  const dim3 grid(2 * p.nQT * p.nbh);
  hipLaunchKernelGGL(fwd_kernel<D>, grid, dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_fwd(const Shape& s, const void* Q, const void* K, const void* V, void* O,
                      float* LSE, hipStream_t st) {
  if (s.D == 128) return launch_fwd_d<128>(s, Q, K, V, O, LSE, st);
  return launch_fwd_d<64>(s, Q, K, V, O, LSE, st);
}

}  // namespace bd
