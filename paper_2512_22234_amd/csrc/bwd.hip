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
// dkdv: one workgroup owns a (batch, KV head, 128-key tile); each of its four
// waves owns 32 keys whose K/V rows stay in registers.  It walks the query
// heads of the GQA group and the query tiles (64 rows) that can see the key
// tile, in the order given by the exact tile classification.  Scores are
// computed as S = Q K^T so each lane owns one key column; P and dS are then
// the B operands of dV^T = dO^T P and dK^T = Q^T dS directly, with Q^T and
// dO^T written to LDS (perm16 order) next to the row-major tiles.
//
// dq: one workgroup owns a (batch, query head, 128-row query tile) like the
// forward; scores are S^T = K Q^T (lane = query), dQ^T = K^T dS^T with K^T
// from the transposed copy.
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
  int L, S, Hq, Hkv, G, nKT, nkv;
  float c;      // scale * log2(e)
  float scale;
};

template <int D>
struct DkvSmem {
  static constexpr int BM = DKV_BM;
  static constexpr int QS = D + 8;   // row-major tile stride (elements)
  static constexpr int TS = BM + 8;  // transposed tile stride
  bf16 q[2][BM * QS];
  bf16 dO[2][BM * QS];
  uint16_t qt[2][D * TS];
  uint16_t dot[2][D * TS];
  float lse2[2][BM];
  float dlt[2][BM];
  int qblk[2][BM];
};

template <int D>
__global__ __launch_bounds__(256, 1) void dkdv_kernel(DkvParams p) {
  constexpr int BM = DKV_BM, BN = DKV_BN;
  constexpr int DS = D / 16, DB = D / 32, QB = BM / 32, PC = BM / 16;
  constexpr int QS = DkvSmem<D>::QS, TS = DkvSmem<D>::TS;
  constexpr int NCH = BM * D / 8 / 256;  // 16-byte chunks per thread, for each of Q and dO
  static_assert(NCH * 256 * 8 == BM * D, "tile must split evenly over 256 threads");
  __shared__ DkvSmem<D> sm;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, g2 = lane >> 5;
  const int L = p.L, S = p.S, N = 2 * L;

  // Clean key tiles first, lowest index (most query tiles) first; the light
  // noisy key tiles last.  Consecutive workgroups are different KV heads.
  const int id = blockIdx.x;
  const int rank = id / p.nkv;
  const int grp = id - rank * p.nkv;  // b * Hkv + hk
  const int kh = rank < p.nKT ? HALF_CLEAN : HALF_NOISY;
  const int j = rank < p.nKT ? rank : rank - p.nKT;
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
  const int T = p.G * per_g;

  u32x4 qst[NCH], dost[NCH];
  float lse_st = 0.f, dlt_st = 0.f;
  int qb_st = QBLK_INVALID;
  auto load_tile = [&](int t) {
    const int g = t / per_g;
    int qh, i;
    ql.at(t - g * per_g, qh, i);
    const size_t bhq = (size_t)b * p.Hq + hk * p.G + g;
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int c = tid + 256 * u;
      const int row = c / (D / 8), col8 = c % (D / 8);
      const int qr = i * BM + row;
      const u32x4 z = {0u, 0u, 0u, 0u};
      const size_t off = (bhq * N + qh * L + qr) * D + col8 * 8;
      qst[u] = qr < L ? ld16(p.Q + off) : z;
      dost[u] = qr < L ? ld16(p.dO + off) : z;
    }
    if (tid < BM) {
      const int qr = i * BM + tid;
      const bool ok = qr < L;
      lse_st = ok ? p.LSE[bhq * N + qh * L + qr] * LOG2E : 0.f;
      dlt_st = ok ? p.delta[bhq * N + qh * L + qr] : 0.f;
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
      const int pr = perm16(row);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = col8 * 8 + e;
        sm.qt[buf][d * TS + pr] = (uint16_t)(qst[u][e >> 1] >> (16 * (e & 1)));
        sm.dot[buf][d * TS + pr] = (uint16_t)(dost[u][e >> 1] >> (16 * (e & 1)));
      }
    }
    if (tid < BM) {
      sm.lse2[buf][tid] = lse_st;
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

  if (T > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();

  for (int t = 0; t < T; ++t) {
    const int buf = t & 1;
    if (t + 1 < T) load_tile(t + 1);
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
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
          const int rr = qb * 32 + 8 * i4 + 4 * g2;
          const f32x4 l4 = *reinterpret_cast<const f32x4*>(&sm.lse2[buf][rr]);
          const f32x4 d4 = *reinterpret_cast<const f32x4*>(&sm.dlt[buf][rr]);
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            float pv = fast_exp2(sacc[qb][4 * i4 + jj] * p.c - l4[jj]);
            if (partial && !visible(qh, sm.qblk[buf][rr + jj], kh, bk)) pv = 0.f;
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
          const bf16x8 ad = *reinterpret_cast<const bf16x8*>(&sm.dot[buf][(db * 32 + l32) * TS + 16 * c + 8 * g2]);
          dvacc[db] = mfma32(ad, pb[c], dvacc[db]);
          const bf16x8 aq = *reinterpret_cast<const bf16x8*>(&sm.qt[buf][(db * 32 + l32) * TS + 16 * c + 8 * g2]);
          dkacc[db] = mfma32(aq, dsb[c], dkacc[db]);
        }
    }
    if (t + 1 < T) store_tile(buf ^ 1);
    __syncthreads();
  }

  if (kvalid) {
    bf16* dkp = p.dK + krow * D + 4 * g2;
    bf16* dvp = p.dV + krow * D + 4 * g2;
    const float sc = p.scale;
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

// ----------------------------------------------------------------------------
struct DqParams {
  const bf16* Q;
  const bf16* K;
  const bf16* Kt;
  const bf16* V;
  const bf16* dO;
  const float* LSE;
  const float* delta;
  bf16* dQ;
  int L, S, Hq, Hkv, G, Lp, nQT, nbh;
  float c;
  float scale;
};

template <int D>
struct DqSmem {
  static constexpr int BN = DQ_BN;
  static constexpr int KS = D + 8;
  static constexpr int VS = BN + 8;
  bf16 k[2][BN * KS];
  bf16 v[2][BN * KS];
  bf16 kt[2][D * VS];
  int kblk[2][BN];
};

template <int D>
__global__ __launch_bounds__(256, 1) void dq_kernel(DqParams p) {
  constexpr int BM = DQ_BM, BN = DQ_BN;
  constexpr int DS = D / 16, DB = D / 32, KB = BN / 32, PC = BN / 16;
  constexpr int KS = DqSmem<D>::KS, VS = DqSmem<D>::VS;
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
  const bf16* Ktp = p.Kt + (size_t)(b * p.Hkv + hk) * D * (2 * p.Lp);

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

  u32x4 kst[NCH], vst[NCH], tst[NCH];
  int kbst = 0;
  auto load_tile = [&](int t) {
    int kh, j;
    kl.at(t, kh, j);
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int c = tid + 256 * u;
      const int row = c / (D / 8), col8 = c % (D / 8);
      const int key = j * BN + row;
      const u32x4 z = {0u, 0u, 0u, 0u};
      const size_t off = kvbase + (size_t)(kh * L + key) * D + col8 * 8;
      kst[u] = key < L ? ld16(p.K + off) : z;
      vst[u] = key < L ? ld16(p.V + off) : z;
      const int d = c / (BN / 8), kc = c % (BN / 8);
      tst[u] = ld16(Ktp + (size_t)d * (2 * p.Lp) + kh * p.Lp + j * BN + kc * 8);
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
      const int d = c / (BN / 8), kc = c % (BN / 8);
      st16(&sm.kt[buf][d * VS + kc * 8], tst[u]);
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
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int* kbp = &sm.kblk[buf][kb * 32 + 8 * i + 4 * g2];
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            const int e = 4 * i + jj;
            float pv = fast_exp2(sacc[kb][e] * p.c - lse2);
            if (partial && !visible(qh, bq, kh, kbp[jj])) pv = 0.f;
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
          const bf16x8 a = lds_bf16x8(&sm.kt[buf][(db * 32 + l32) * VS + 16 * c + 8 * g2]);
          dqacc[db] = mfma32(a, dsb[c], dqacc[db]);
        }
    }
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
                         const float* LSE, const float* delta, void* dK, void* dV, hipStream_t st) {
  DkvParams p;
  p.Q = static_cast<const bf16*>(Q);
  p.K = static_cast<const bf16*>(K);
  p.V = static_cast<const bf16*>(V);
  p.dO = static_cast<const bf16*>(dO);
  p.LSE = LSE;
  p.delta = delta;
  p.dK = static_cast<bf16*>(dK);
  p.dV = static_cast<bf16*>(dV);
  p.L = s.L;
  p.S = s.S;
  p.Hq = s.Hq;
  p.Hkv = s.Hkv;
  p.G = s.G;
  p.nKT = cdiv(s.L, DKV_BN);
  p.nkv = s.B * s.Hkv;
  p.c = s.scale * LOG2E;
  p.scale = s.scale;
  const dim3 grid(2 * p.nKT * p.nkv);
  hipLaunchKernelGGL(dkdv_kernel<D>, grid, dim3(256), 0, st, p);
  return hipGetLastError();
}

template <int D>
hipError_t launch_dq_d(const Shape& s, const void* Q, const void* K, const void* Kt, const void* V,
                       const void* dO, const float* LSE, const float* delta, void* dQ, hipStream_t st) {
  DqParams p;
  p.Q = static_cast<const bf16*>(Q);
  p.K = static_cast<const bf16*>(K);
  p.Kt = static_cast<const bf16*>(Kt);
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
  p.Lp = s.Lp;
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
                           const float* LSE, const float* delta, void* dK, void* dV, hipStream_t st) {
  if (s.D == 128) return launch_dkdv_d<128>(s, Q, K, V, dO, LSE, delta, dK, dV, st);
  return launch_dkdv_d<64>(s, Q, K, V, dO, LSE, delta, dK, dV, st);
}

hipError_t launch_bwd_dq(const Shape& s, const void* Q, const void* K, const void* Kt, const void* V,
                         const void* dO, const float* LSE, const float* delta, void* dQ, hipStream_t st) {
  if (s.D == 128) return launch_dq_d<128>(s, Q, K, Kt, V, dO, LSE, delta, dQ, st);
  return launch_dq_d<64>(s, Q, K, Kt, V, dO, LSE, delta, dQ, st);
}

}  // namespace bd
