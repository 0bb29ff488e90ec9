// Backward pass of block-diffusion masked attention for gfx950: the
// vector-Jacobian product of softmax attention under the mask of Eq. 1 / Eq. 2
// (DiRL Section 4.1), with no atomics, so results are bitwise reproducible.
//
//   Delta = rowsum(dO * O)                              (bwd_pre)
//   P     = exp(scale Q K^T - LSE) on visible pairs
//   dV    = P^T dO,  dP = dO V^T,  dS = P * (dP - Delta)
//   dK    = scale dS^T Q                                (dkdv, key-tile major)
//   dQ    = scale dS K                                  (dq, query-tile major)
//
// dkdv: a workgroup owns a (batch, KV head, 128-key tile); each of its four
// waves owns 32 keys whose K/V rows stay in registers.  It walks the query
// heads of the GQA group and the 64-row query tiles that can see the key tile
// (the exact tile classification gives the list).  Scores are S = Q K^T so
// each lane owns one key column; P and dS are then directly the B operands of
// dV^T = dO^T P and dK^T = Q^T dS, whose A operands come from the row-major Q
// and dO tiles through the transposing LDS read.  Work per clean key tile
// shrinks linearly with its position, so each clean tile's walk is split into
// two halves run by two workgroups that write float32 partial sums; a combine
// kernel adds the two halves in a fixed order.  Noisy key tiles (seen only by
// their own block's noisy queries) are done by one workgroup each.
//
// dq: a workgroup owns a (batch, query head, 128-row query tile) like the
// forward; scores are S^T = K Q^T (lane = query) and dQ^T = K^T dS^T with K^T
// read from the row-major K tile through the transposing LDS read.
#include "device.hpp"
#include "kernels.hpp"

namespace bd {
namespace {

// ----------------------------------------------------------------------------
// Delta = rowsum(dO * O) in fp32; D/8 consecutive lanes share one row.
template <int D>
__global__ __launch_bounds__(256) void bwd_pre_kernel(const bf16* __restrict__ O,
                                                      const bf16* __restrict__ dO,
                                                      float* __restrict__ delta, size_t rows) {
  constexpr int TPR = D / 8;
  const size_t gid = (size_t)blockIdx.x * 256 + threadIdx.x;
  const size_t row = gid / TPR;
  const int part = (int)(gid % TPR);
  float acc = 0.f;
  if (row < rows) {
    const bf16x8 o = *reinterpret_cast<const bf16x8*>(O + row * D + part * 8);
    const bf16x8 g = *reinterpret_cast<const bf16x8*>(dO + row * D + part * 8);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc += (float)o[e] * (float)g[e];
  }
#pragma unroll
  for (int off = TPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (row < rows && part == 0) delta[row] = acc;
}

// ----------------------------------------------------------------------------
struct DkvParams {
  const bf16* Q;
  const bf16* K;
  const bf16* V;
  const bf16* dO;
  const float* LSE;
  const float* delta;
  bf16* dK;
  bf16* dV;
  float* part;  // [2 halves][2 (dK, dV)][B*Hkv][L][D] partial sums of clean key tiles
  int L, S, Hq, Hkv, G, nKT, nkv;
  float c;      // scale * log2(e)
  float scale;
};

template <int D>
struct DkvSmem {
  static constexpr int BM = DKV_BM;
  static constexpr int QS = D + 8;  // row stride (elements)
  bf16 q[2][BM * QS];
  bf16 dO[2][BM * QS];
  alignas(16) float lse2[2][BM];
  alignas(16) float dlt[2][BM];
  alignas(16) int qblk[2][BM];
};

template <int D>
__global__ __launch_bounds__(256, 1) void dkdv_kernel(DkvParams p) {
  constexpr int BM = DKV_BM, BN = DKV_BN;
  constexpr int DS = D / 16, DB = D / 32, QB = BM / 32, PC = BM / 16;
  constexpr int QS = DkvSmem<D>::QS;
  constexpr int NCH = BM * D / 8 / 256;  // 16-byte chunks per thread, for each of Q and dO
  static_assert(NCH * 256 * 8 == BM * D, "tile must split evenly over 256 threads");
  __shared__ DkvSmem<D> sm;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, g2 = lane >> 5;
  const int L = p.L, S = p.S, N = 2 * L;

  // Items: clean key tiles in ascending index (most work first), each as two
  // halves of its walk; then noisy key tiles, one item each.  Consecutive
  // workgroups are different KV heads.
  const int id = blockIdx.x;
  const int rank = id / p.nkv;
  const int grp = id - rank * p.nkv;  // b * Hkv + hk
  const bool clean = rank < 2 * p.nKT;
  const int kh = clean ? HALF_CLEAN : HALF_NOISY;
  const int j = clean ? (rank >> 1) : rank - 2 * p.nKT;
  const int split = clean ? (rank & 1) : 0;
  const int b = grp / p.Hkv, hk = grp - b * p.Hkv;
  const int k0 = j * BN, k1 = imin(L, k0 + BN);

  const int kk = k0 + w * 32 + l32;  // this lane's key (local to its half)
  const bool kvalid = kk < k1;
  const int bk = kvalid ? kk / S : KBLK_INVALID;
  const size_t krow = (size_t)grp * N + kh * L + kk;

  bf16x8 kreg[DS], vreg[DS];
#pragma unroll
  for (int s = 0; s < DS; ++s) {
    kreg[s] = kvalid ? *reinterpret_cast<const bf16x8*>(p.K + krow * D + 16 * s + 8 * g2) : zero_bf16x8();
    vreg[s] = kvalid ? *reinterpret_cast<const bf16x8*>(p.V + krow * D + 16 * s + 8 * g2) : zero_bf16x8();
  }

  const QueryTileList ql = query_tiles_for_key_tile(kh, j, L, S, BM, BN);
  const int per_g = ql.count();
  const int Tall = p.G * per_g;
  const int t0 = clean ? (split * Tall) / 2 : 0;
  const int t1 = clean ? ((split + 1) * Tall) / 2 : Tall;

  u32x4 qst[NCH], dost[NCH];
  float lse_st = 0.f, dlt_st = 0.f;
  int qb_st = QBLK_INVALID;
  auto load_tile = [&](int t) {
    const int g = t / per_g;
    int qh, i;
    ql.at(t - g * per_g, qh, i);
    const size_t bhq = (size_t)b * p.Hq + hk * p.G + g;
    const size_t hbase = (bhq * N + qh * L) * D;
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int c = tid + 256 * u;
      const int row = c / (D / 8), col8 = c % (D / 8);
      qst[u] = ld16_rows(p.Q + hbase, i * BM + row, L, D, col8 * 8);
      dost[u] = ld16_rows(p.dO + hbase, i * BM + row, L, D, col8 * 8);
    }
    if (tid < BM) {
      const int qr = i * BM + tid;
      const bool ok = qr < L;
      const size_t rr = bhq * N + qh * L + (ok ? qr : L - 1);
      lse_st = p.LSE[rr];  // rows past the end are masked (qblk invalid)
      dlt_st = p.delta[rr];
      qb_st = ok ? qr / S : QBLK_INVALID;
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int c = tid + 256 * u;
      const int row = c / (D / 8), col8 = c % (D / 8);
      st16(&sm.q[buf][row * QS + col8 * 8], qst[u]);
      st16(&sm.dO[buf][row * QS + col8 * 8], dost[u]);
    }
    if (tid < BM) {
      sm.lse2[buf][tid] = lse_st * LOG2E;
      sm.dlt[buf][tid] = dlt_st;
      sm.qblk[buf][tid] = qb_st;
    }
  };

  f32x16 dkacc[DB], dvacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      dkacc[db][e] = 0.f;
      dvacc[db][e] = 0.f;
    }

  if (t0 < t1) {
    load_tile(t0);
    store_tile(0);
  }
  wait_global_loads();  // K/V rows are in registers; the loop only waits on its own prefetch
  __syncthreads();

  for (int t = t0; t < t1; ++t) {
    const int buf = (t - t0) & 1;
    if (t + 1 < t1) load_tile(t + 1);
    const int g = t / per_g;
    int qh, i;
    ql.at(t - g * per_g, qh, i);
    const int q0 = i * BM, q1 = imin(L, q0 + BM);
    const int cls = classify_pair(qh, q0, q1, kh, k0, k1, S, (q1 - q0) == BM && (k1 - k0) == BN);
    if (cls != TILE_EMPTY) {
      f32x16 sacc[QB], dpacc[QB];
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          sacc[qb][e] = 0.f;
          dpacc[qb][e] = 0.f;
        }
      // S[q][key] = sum_d Q[q][d] K[key][d];  dP[q][key] = sum_d dO[q][d] V[key][d]
#pragma unroll
      for (int s = 0; s < DS; ++s)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          const bf16x8 aq = lds_bf16x8(&sm.q[buf][(qb * 32 + l32) * QS + 16 * s + 8 * g2]);
          sacc[qb] = mfma32(aq, kreg[s], sacc[qb]);
          const bf16x8 ad = lds_bf16x8(&sm.dO[buf][(qb * 32 + l32) * QS + 16 * s + 8 * g2]);
          dpacc[qb] = mfma32(ad, vreg[s], dpacc[qb]);
        }
      const bool partial = cls == TILE_PARTIAL;
      const BlockWindow win = query_window(qh, kh, bk);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
          const int rr = qb * 32 + 8 * i4 + 4 * g2;
          const f32x4 l4 = *reinterpret_cast<const f32x4*>(&sm.lse2[buf][rr]);
          const f32x4 d4 = *reinterpret_cast<const f32x4*>(&sm.dlt[buf][rr]);
          const int4 qb4 = *reinterpret_cast<const int4*>(&sm.qblk[buf][rr]);
          const int qbv[4] = {qb4.x, qb4.y, qb4.z, qb4.w};
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            float pv = fast_exp2(sacc[qb][4 * i4 + jj] * p.c - l4[jj]);
            pv = (!partial || win.has(qbv[jj])) ? pv : 0.f;
            dpacc[qb][4 * i4 + jj] = pv * (dpacc[qb][4 * i4 + jj] - d4[jj]);
            sacc[qb][4 * i4 + jj] = pv;
          }
        }
      bf16x8 pb[PC], dsb[PC];
#pragma unroll
      for (int c = 0; c < PC; ++c) {
        pb[c] = pack8(sacc[c >> 1], 8 * (c & 1));
        dsb[c] = pack8(dpacc[c >> 1], 8 * (c & 1));
      }
      // dV^T[d][key] += sum_q dO^T[d][q] P[q][key];  dK^T[d][key] += sum_q Q^T[d][q] dS[q][key]
#pragma unroll
      for (int c = 0; c < PC; ++c)
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const bf16x8 ad = lds_read_tr(sm.dO[buf], QS, 16 * c, db * 32, lane);
          dvacc[db] = mfma32(ad, pb[c], dvacc[db]);
          const bf16x8 aq = lds_read_tr(sm.q[buf], QS, 16 * c, db * 32, lane);
          dkacc[db] = mfma32(aq, dsb[c], dkacc[db]);
        }
    }
    compute_fence();
    if (t + 1 < t1) store_tile(buf ^ 1);
    __syncthreads();
  }

  if (!kvalid) return;
  const float sc = p.scale;
  if (clean) {
    // float32 partial sums; the combine kernel adds the two halves
    const size_t plane = (size_t)p.nkv * L * D;
    float* pk = p.part + (size_t)(2 * split) * plane + ((size_t)grp * L + kk) * D + 4 * g2;
    float* pv = pk + plane;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f32x4 vk = {dkacc[db][4 * i] * sc, dkacc[db][4 * i + 1] * sc, dkacc[db][4 * i + 2] * sc,
                          dkacc[db][4 * i + 3] * sc};
        const f32x4 vv = {dvacc[db][4 * i], dvacc[db][4 * i + 1], dvacc[db][4 * i + 2], dvacc[db][4 * i + 3]};
        *reinterpret_cast<f32x4*>(pk + db * 32 + 8 * i) = vk;
        *reinterpret_cast<f32x4*>(pv + db * 32 + 8 * i) = vv;
      }
  } else {
    bf16* dkp = p.dK + krow * D + 4 * g2;
    bf16* dvp = p.dV + krow * D + 4 * g2;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        st_bf16x4(dkp + db * 32 + 8 * i, dkacc[db][4 * i] * sc, dkacc[db][4 * i + 1] * sc,
                  dkacc[db][4 * i + 2] * sc, dkacc[db][4 * i + 3] * sc);
        st_bf16x4(dvp + db * 32 + 8 * i, dvacc[db][4 * i], dvacc[db][4 * i + 1], dvacc[db][4 * i + 2],
                  dvacc[db][4 * i + 3]);
      }
  }
}

// dK/dV of the clean half = half0 + half1 (fixed order), rounded to bf16.
// One thread per 4 consecutive features.
__global__ __launch_bounds__(256) void dkdv_combine_kernel(const float* __restrict__ part, bf16* __restrict__ dK,
                                                           bf16* __restrict__ dV, int nkv, int L, int D) {
  const size_t plane = (size_t)nkv * L * D;
  const size_t quads = plane / 4;
  const size_t stride = (size_t)gridDim.x * 256;
  for (size_t qd = (size_t)blockIdx.x * 256 + threadIdx.x; qd < quads; qd += stride) {
    const size_t e = qd * 4;
    const size_t row = e / D;  // grp * L + key
    const size_t grp = row / L, key = row - grp * L;
    const size_t out = ((grp * 2 + 1) * L + key) * D + (e - row * D);
    const f32x4 k0 = *reinterpret_cast<const f32x4*>(part + e);
    const f32x4 v0 = *reinterpret_cast<const f32x4*>(part + plane + e);
    const f32x4 k1 = *reinterpret_cast<const f32x4*>(part + 2 * plane + e);
    const f32x4 v1 = *reinterpret_cast<const f32x4*>(part + 3 * plane + e);
    st_bf16x4(dK + out, k0[0] + k1[0], k0[1] + k1[1], k0[2] + k1[2], k0[3] + k1[3]);
    st_bf16x4(dV + out, v0[0] + v1[0], v0[1] + v1[1], v0[2] + v1[2], v0[3] + v1[3]);
  }
}

// ----------------------------------------------------------------------------
struct DqParams {
  const bf16* Q;
  const bf16* K;
  const bf16* V;
  const bf16* dO;
  const float* LSE;
  const float* delta;
  bf16* dQ;
  int L, S, Hq, Hkv, G, nQT, nbh;
  float c;
  float scale;
};

template <int D>
struct DqSmem {
  static constexpr int BN = DQ_BN;
  static constexpr int KS = D + 8;
  bf16 k[2][BN * KS];
  bf16 v[2][BN * KS];
  alignas(16) int kblk[2][BN];
};

template <int D>
__global__ __launch_bounds__(256, 2) void dq_kernel(DqParams p) {
  constexpr int BM = DQ_BM, BN = DQ_BN;
  constexpr int DS = D / 16, DB = D / 32, KB = BN / 32, PC = BN / 16;
  constexpr int KS = DqSmem<D>::KS;
  constexpr int NCH = BN * D / 8 / 256;
  static_assert(NCH * 256 * 8 == BN * D, "tile must split evenly over 256 threads");
  __shared__ DqSmem<D> sm;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, g2 = lane >> 5;
  const int L = p.L, S = p.S, N = 2 * L;

  const int id = blockIdx.x;
  const int rank = id / p.nbh;
  const int bh = xcd_head_remap(id - rank * p.nbh, p.nbh, p.G);
  const int qi = p.nQT - 1 - (rank >> 1);
  const int qh = rank & 1;
  const int b = bh / p.Hq, hq = bh - b * p.Hq, hk = hq / p.G;
  const int q0 = qi * BM, q1 = imin(L, q0 + BM);

  const size_t kvbase = (size_t)(b * p.Hkv + hk) * N * D;

  const int r = q0 + w * 32 + l32;
  const bool qvalid = r < q1;
  const int bq = qvalid ? r / S : QBLK_INVALID;
  const int prow = qh * L + r;
  const size_t qrow = (size_t)bh * N + prow;

  bf16x8 qreg[DS], doreg[DS];
#pragma unroll
  for (int s = 0; s < DS; ++s) {
    qreg[s] = qvalid ? *reinterpret_cast<const bf16x8*>(p.Q + qrow * D + 16 * s + 8 * g2) : zero_bf16x8();
    doreg[s] = qvalid ? *reinterpret_cast<const bf16x8*>(p.dO + qrow * D + 16 * s + 8 * g2) : zero_bf16x8();
  }
  const float lse2 = qvalid ? p.LSE[qrow] * LOG2E : 0.f;
  const float dlt = qvalid ? p.delta[qrow] : 0.f;

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

  f32x16 dqacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) dqacc[db][e] = 0.f;

  if (T > 0) {
    load_tile(0);
    store_tile(0);
  }
  wait_global_loads();  // Q/dO rows are in registers; the loop only waits on its own prefetch
  __syncthreads();

  for (int t = 0; t < T; ++t) {
    const int buf = t & 1;
    if (t + 1 < T) load_tile(t + 1);
    int kh, j;
    kl.at(t, kh, j);
    const int k0 = j * BN, k1 = imin(L, k0 + BN);
    const int cls = classify_pair(qh, q0, q1, kh, k0, k1, S, (q1 - q0) == BM && (k1 - k0) == BN);
    if (cls != TILE_EMPTY) {
      f32x16 sacc[KB], dpacc[KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          sacc[kb][e] = 0.f;
          dpacc[kb][e] = 0.f;
        }
      // S^T[key][q] = sum_d K[key][d] Q[q][d];  dP^T[key][q] = sum_d V[key][d] dO[q][d]
#pragma unroll
      for (int s = 0; s < DS; ++s)
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          const bf16x8 ak = lds_bf16x8(&sm.k[buf][(kb * 32 + l32) * KS + 16 * s + 8 * g2]);
          sacc[kb] = mfma32(ak, qreg[s], sacc[kb]);
          const bf16x8 av = lds_bf16x8(&sm.v[buf][(kb * 32 + l32) * KS + 16 * s + 8 * g2]);
          dpacc[kb] = mfma32(av, doreg[s], dpacc[kb]);
        }
      const bool partial = cls == TILE_PARTIAL;
      const BlockWindow win = key_window(qh, kh, bq);
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int4 kb4 = *reinterpret_cast<const int4*>(&sm.kblk[buf][kb * 32 + 8 * i + 4 * g2]);
          const int kbv[4] = {kb4.x, kb4.y, kb4.z, kb4.w};
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            const int e = 4 * i + jj;
            float pv = fast_exp2(sacc[kb][e] * p.c - lse2);
            pv = (!partial || win.has(kbv[jj])) ? pv : 0.f;
            sacc[kb][e] = pv * (dpacc[kb][e] - dlt);
          }
        }
      bf16x8 dsb[PC];
#pragma unroll
      for (int c = 0; c < PC; ++c) dsb[c] = pack8(sacc[c >> 1], 8 * (c & 1));
      // dQ^T[d][q] += sum_key K^T[d][key] dS^T[key][q]
#pragma unroll
      for (int c = 0; c < PC; ++c)
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const bf16x8 a = lds_read_tr(sm.k[buf], KS, 16 * c, db * 32, lane);
          dqacc[db] = mfma32(a, dsb[c], dqacc[db]);
        }
    }
    compute_fence();
    if (t + 1 < T) store_tile(buf ^ 1);
    __syncthreads();
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
hipError_t launch_pre_d(const Shape& s, const void* O, const void* dO, float* delta, hipStream_t st) {
  const size_t rows = (size_t)s.B * s.Hq * 2 * s.L;
  const size_t threads = rows * (D / 8);
  const dim3 grid((unsigned)((threads + 255) / 256));
  hipLaunchKernelGGL(bwd_pre_kernel<D>, grid, dim3(256), 0, st, static_cast<const bf16*>(O),
                     static_cast<const bf16*>(dO), delta, rows);
  return hipGetLastError();
}

template <int D>
hipError_t launch_dkdv_d(const Shape& s, const void* Q, const void* K, const void* V, const void* dO,
                         const float* LSE, const float* delta, void* dK, void* dV, float* part, hipStream_t st) {
  DkvParams p;
  p.Q = static_cast<const bf16*>(Q);
  p.K = static_cast<const bf16*>(K);
  p.V = static_cast<const bf16*>(V);
  p.dO = static_cast<const bf16*>(dO);
  p.LSE = LSE;
  p.delta = delta;
  p.dK = static_cast<bf16*>(dK);
  p.dV = static_cast<bf16*>(dV);
  p.part = part;
  p.L = s.L;
  p.S = s.S;
  p.Hq = s.Hq;
  p.Hkv = s.Hkv;
  p.G = s.G;
  p.nKT = cdiv(s.L, DKV_BN);
  p.nkv = s.B * s.Hkv;
  p.c = s.scale * LOG2E;
  p.scale = s.scale;
  const dim3 grid(3 * p.nKT * p.nkv);
  hipLaunchKernelGGL(dkdv_kernel<D>, grid, dim3(256), 0, st, p);
  return hipGetLastError();
}

template <int D>
hipError_t launch_dq_d(const Shape& s, const void* Q, const void* K, const void* V, const void* dO,
                       const float* LSE, const float* delta, void* dQ, hipStream_t st) {
  DqParams p;
  p.Q = static_cast<const bf16*>(Q);
  p.K = static_cast<const bf16*>(K);
  p.V = static_cast<const bf16*>(V);
  p.dO = static_cast<const bf16*>(dO);
  p.LSE = LSE;
  p.delta = delta;
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
  hipLaunchKernelGGL(dq_kernel<D>, grid, dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bwd_pre(const Shape& s, const void* O, const void* dO, float* delta, hipStream_t st) {
  if (s.D == 128) return launch_pre_d<128>(s, O, dO, delta, st);
  return launch_pre_d<64>(s, O, dO, delta, st);
}

hipError_t launch_bwd_dkdv(const Shape& s, const void* Q, const void* K, const void* V, const void* dO,
                           const float* LSE, const float* delta, void* dK, void* dV, float* part,
                           hipStream_t st) {
  if (s.D == 128) return launch_dkdv_d<128>(s, Q, K, V, dO, LSE, delta, dK, dV, part, st);
  return launch_dkdv_d<64>(s, Q, K, V, dO, LSE, delta, dK, dV, part, st);
}

hipError_t launch_bwd_dkdv_combine(const Shape& s, const float* part, void* dK, void* dV, hipStream_t st) {
  const int nkv = s.B * s.Hkv;
  const size_t quads = (size_t)nkv * s.L * s.D / 4;
  size_t blocks = (quads + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(dkdv_combine_kernel, dim3((unsigned)blocks), dim3(256), 0, st, part, static_cast<bf16*>(dK),
                     static_cast<bf16*>(dV), nkv, s.L, s.D);
  return hipGetLastError();
}

hipError_t launch_bwd_dq(const Shape& s, const void* Q, const void* K, const void* V, const void* dO,
                         const float* LSE, const float* delta, void* dQ, hipStream_t st) {
  if (s.D == 128) return launch_dq_d<128>(s, Q, K, V, dO, LSE, delta, dQ, st);
  return launch_dq_d<64>(s, Q, K, V, dO, LSE, delta, dQ, st);
}

}  // namespace bd
