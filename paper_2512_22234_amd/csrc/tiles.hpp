// Tile geometry and exact tile classification for the block-diffusion mask.
//
// Packed sequence [x_t | x_0] of 2L positions; each half is cut into tiles
// independently ("half-local" tiles, the last one shorter when the tile size
// does not divide L), so every tile lies in one half and the quadrant of a
// (query tile, key tile) pair is fixed.  Inside a half the block index
// b = local_position div S is non-decreasing, so the block-index range of a
// tile is [first div S, last div S] and the class of a pair follows from the
// two ranges alone (DiRL Section 4.1 with the rules of Eq. 1 and Eq. 2):
//
//   quadrant      visible pair when     FULL iff            EMPTY iff
//   noisy-noisy   bk == bq              qlo=qhi=klo=khi     qhi<klo or khi<qlo
//   noisy-clean   bk <  bq              khi <  qlo          klo >= qhi
//   clean-clean   bk <= bq              khi <= qlo          klo >  qhi
//   clean-noisy   never                 never               always
//
// A pair that is not EMPTY is downgraded from FULL to PARTIAL when either tile
// is short (ragged end of a half), so that a FULL tile can run with no
// per-element test at all.
//
// This header is plain C++ apart from the host/device qualifiers, so the host
// classifier exported by the library and the kernels use the same code.
#pragma once

#ifdef __HIPCC__
#define BD_HD __host__ __device__ inline
#else
#define BD_HD inline
#endif

namespace bd {

enum { TILE_EMPTY = 0, TILE_FULL = 1, TILE_PARTIAL = 2 };
enum { HALF_NOISY = 0, HALF_CLEAN = 1 };

BD_HD int cdiv(int a, int b) { return (a + b - 1) / b; }
BD_HD int imin(int a, int b) { return a < b ? a : b; }
BD_HD int imax(int a, int b) { return a > b ? a : b; }

// Is key (half kh, block bk) visible from query (half qh, block bq)?
BD_HD bool visible(int qh, int bq, int kh, int bk) {
  if (qh == HALF_NOISY) return kh == HALF_NOISY ? bk == bq : bk < bq;
  return kh == HALF_CLEAN && bk <= bq;
}

// Class of the pair (query rows [q0,q1) of half qh, keys [k0,k1) of half kh);
// local indices, both ranges non-empty.  full_size: both tiles full-sized.
BD_HD int classify_pair(int qh, int q0, int q1, int kh, int k0, int k1, int S, bool full_size) {
  const int qlo = q0 / S, qhi = (q1 - 1) / S, klo = k0 / S, khi = (k1 - 1) / S;
  int cls;
  if (qh == HALF_NOISY && kh == HALF_NOISY) {
    if (qhi < klo || khi < qlo) return TILE_EMPTY;
    cls = (qlo == qhi && klo == khi && qlo == klo) ? TILE_FULL : TILE_PARTIAL;
  } else if (qh == HALF_NOISY) {
    if (klo >= qhi) return TILE_EMPTY;
    cls = (khi < qlo) ? TILE_FULL : TILE_PARTIAL;
  } else if (kh == HALF_CLEAN) {
    if (klo > qhi) return TILE_EMPTY;
    cls = (khi <= qlo) ? TILE_FULL : TILE_PARTIAL;
  } else {
    return TILE_EMPTY;
  }
  if (cls == TILE_FULL && !full_size) cls = TILE_PARTIAL;
  return cls;
}

// Division-free forms of classify_pair used inside the kernels.  For a fixed
// tile whose block range is [lo, hi], pass A = lo*S and B = hi*S (the first
// positions of its first and last block); the moving tile is [m0, m1).  The
// comparisons are those of classify_pair with both sides multiplied by S.
//
// Fixed query tile (half qh), moving key tile (half kh).
BD_HD int classify_vs_query_tile(int qh, int A, int B, int S, int kh, int k0, int k1, bool full_size) {
  int cls;
  if (qh == HALF_NOISY && kh == HALF_NOISY) {
    if (k0 >= B + S || k1 <= A) return TILE_EMPTY;
    cls = (A == B && k0 >= A && k1 <= A + S) ? TILE_FULL : TILE_PARTIAL;
  } else if (qh == HALF_NOISY) {
    if (k0 >= B) return TILE_EMPTY;
    cls = (k1 <= A) ? TILE_FULL : TILE_PARTIAL;
  } else if (kh == HALF_CLEAN) {
    if (k0 >= B + S) return TILE_EMPTY;
    cls = (k1 <= A + S) ? TILE_FULL : TILE_PARTIAL;
  } else {
    return TILE_EMPTY;
  }
  if (cls == TILE_FULL && !full_size) cls = TILE_PARTIAL;
  return cls;
}
// Fixed key tile (half kh), moving query tile (half qh).
BD_HD int classify_vs_key_tile(int kh, int A, int B, int S, int qh, int q0, int q1, bool full_size) {
  int cls;
  if (qh == HALF_NOISY && kh == HALF_NOISY) {
    if (q1 <= A || q0 >= B + S) return TILE_EMPTY;
    cls = (A == B && q0 >= A && q1 <= A + S) ? TILE_FULL : TILE_PARTIAL;
  } else if (qh == HALF_NOISY) {
    if (q1 <= A + S) return TILE_EMPTY;
    cls = (q0 >= B + S) ? TILE_FULL : TILE_PARTIAL;
  } else if (kh == HALF_CLEAN) {
    if (q1 <= A) return TILE_EMPTY;
    cls = (q0 >= B) ? TILE_FULL : TILE_PARTIAL;
  } else {
    return TILE_EMPTY;
  }
  if (cls == TILE_FULL && !full_size) cls = TILE_PARTIAL;
  return cls;
}

// The FULL test of classify_vs_key_tile / classify_vs_query_tile for a
// visited pair, reduced to two comparisons per step: with one tile fixed, a
// moving tile [x0, x0 + n) of half h (n its full size) is FULL iff
// lo(h) <= x0 and x0 + n <= hi(h); hi < 0 means never.  A FULL tile is
// full-sized, so the moving tile's own size check is x0 + n <= L.
struct FullRange {
  int lo_n, hi_n, lo_c, hi_c;  // for a moving tile in the noisy / clean half
  BD_HD bool full(int half, int x0, int n) const {
    return half == HALF_NOISY ? (x0 >= lo_n && x0 + n <= hi_n) : (x0 >= lo_c && x0 + n <= hi_c);
  }
  // With the fixed tile a query tile: the number of leading clean key tiles
  // of size n (the walk's first tiles) that are FULL.
  BD_HD int full_prefix(int n) const { return lo_c == 0 && hi_c > 0 ? hi_c / n : 0; }
};
// Fixed key tile [k0, k1) of half kh (full-sized iff k1 - k0 == BN); moving query tiles.
BD_HD FullRange full_range_vs_key_tile(int kh, int k0, int k1, int L, int S, int BN) {
  const int A = (k0 / S) * S, B = ((k1 - 1) / S) * S;
  const bool kfull = (k1 - k0) == BN;
  FullRange r;
  if (kh == HALF_CLEAN) {
    r.lo_n = B + S;  // noisy queries of later blocks only
    r.hi_n = kfull ? L : -1;
    r.lo_c = B;      // clean queries of the same or later blocks
    r.hi_c = kfull ? L : -1;
  } else {
    r.lo_n = A;      // noisy queries of the key tile's own (single) block
    r.hi_n = (kfull && A == B) ? imin(L, A + S) : -1;
    r.lo_c = 0;
    r.hi_c = -1;     // clean queries never see noisy keys
  }
  return r;
}
// Fixed query tile [q0, q1) of half qh (full-sized iff q1 - q0 == BM); moving key tiles.
BD_HD FullRange full_range_vs_query_tile(int qh, int q0, int q1, int L, int S, int BM) {
  const int A = (q0 / S) * S, B = ((q1 - 1) / S) * S;
  const bool qfull = (q1 - q0) == BM;
  FullRange r;
  if (qh == HALF_NOISY) {
    r.lo_n = A;      // noisy keys of the query tile's own (single) block
    r.hi_n = (qfull && A == B) ? imin(L, A + S) : -1;
    r.lo_c = 0;      // clean keys of strictly earlier blocks
    r.hi_c = qfull ? A : -1;
  } else {
    r.lo_n = 0;
    r.hi_n = -1;     // clean queries never see noisy keys
    r.lo_c = 0;      // clean keys of the same or earlier blocks
    r.hi_c = qfull ? imin(L, A + S) : -1;
  }
  return r;
}

// Visible positions of the other half for one row, as a half-open window of
// local positions [lo, hi) (empty when lo == hi).  pos_block_start = b*S for
// the row's block b.  Past-the-end rows pass valid = false.
struct PosWindow {
  int lo, hi;
};
// For a query (block start a = bq*S) looking at keys of half kh.
BD_HD PosWindow keys_visible_from(int qh, int kh, int a, int L, int S, bool valid) {
  if (!valid) return {0, 0};
  if (qh == HALF_NOISY) return kh == HALF_NOISY ? PosWindow{a, imin(L, a + S)} : PosWindow{0, a};
  return kh == HALF_CLEAN ? PosWindow{0, imin(L, a + S)} : PosWindow{0, 0};
}
// For a key (block start a = bk*S) seen by queries of half qh.
BD_HD PosWindow queries_seeing(int kh, int qh, int a, int L, int S, bool valid) {
  if (!valid) return {0, 0};
  if (qh == HALF_NOISY) return kh == HALF_NOISY ? PosWindow{a, imin(L, a + S)} : PosWindow{imin(L, a + S), L};
  return kh == HALF_CLEAN ? PosWindow{a, L} : PosWindow{0, 0};
}

// Unions of those windows over a run of consecutive positions [r0, r1) of one
// half (empty when r0 >= r1).  Each row's window is an interval and the
// windows of consecutive rows are either nested or adjacent, so the union is
// again one interval, and it is exactly the set of positions that some row of
// the run sees (or is seen by).
// Keys of half kh visible from some query of [r0, r1) in half qh.
BD_HD PosWindow wave_keys_visible(int qh, int kh, int r0, int r1, int L, int S) {
  if (r0 >= r1) return {0, 0};
  const int a0 = (r0 / S) * S, a1 = ((r1 - 1) / S) * S;  // block starts of the first and last row
  if (qh == HALF_NOISY) return kh == HALF_NOISY ? PosWindow{a0, imin(L, a1 + S)} : PosWindow{0, a1};
  return kh == HALF_CLEAN ? PosWindow{0, imin(L, a1 + S)} : PosWindow{0, 0};
}
// Queries of half qh that see some key of [r0, r1) in half kh.
BD_HD PosWindow wave_queries_seeing(int kh, int qh, int r0, int r1, int L, int S) {
  if (r0 >= r1) return {0, 0};
  const int a0 = (r0 / S) * S, a1 = ((r1 - 1) / S) * S;
  if (qh == HALF_NOISY)
    return kh == HALF_NOISY ? PosWindow{a0, imin(L, a1 + S)} : PosWindow{imin(L, a0 + S), L};
  return kh == HALF_CLEAN ? PosWindow{a0, L} : PosWindow{0, 0};
}

// The queries of each half that see some key of the group [r0, min(r0 + 32,
// k1)) of half kh (one wave's keys in the dK/dV kernel; empty past k1).
struct KeyGroupSight {
  PosWindow n, c;
  BD_HD KeyGroupSight(int kh, int r0, int k1, int L, int S)
      : n(wave_queries_seeing(kh, HALF_NOISY, r0, imin(k1, r0 + 32), L, S)),
        c(wave_queries_seeing(kh, HALF_CLEAN, r0, imin(k1, r0 + 32), L, S)) {}
  // whether some query of [q0, min(L, q0 + nq)) of half qh sees one of the keys
  BD_HD bool sees(int qh, int q0, int nq, int L) const {
    const PosWindow v = qh == HALF_NOISY ? n : c;
    return v.lo < v.hi && q0 < v.hi && imin(L, q0 + nq) > v.lo;
  }
};

// Key tiles visited by query tile (qh, i): clean key tiles [0, nclean) then,
// for a noisy query tile, noisy key tiles [noisy0, noisy0 + nnoisy).
struct KeyTileList {
  int nclean, noisy0, nnoisy;
  BD_HD int count() const { return nclean + nnoisy; }
  // t-th visited key tile: half and index
  BD_HD void at(int t, int& kh, int& j) const {
    if (t < nclean) { kh = HALF_CLEAN; j = t; }
    else { kh = HALF_NOISY; j = noisy0 + (t - nclean); }
  }
};

BD_HD KeyTileList key_tiles_for_query_tile(int qh, int i, int L, int S, int BM, int BN) {
  const int nKT = cdiv(L, BN);
  const int q0 = i * BM, q1 = imin(L, q0 + BM);
  const int qlo = q0 / S, qhi = (q1 - 1) / S;
  KeyTileList r;
  if (qh == HALF_NOISY) {
    // clean key tile j is visible iff its first block < qhi, i.e. j*BN < qhi*S
    r.nclean = imin(nKT, cdiv(qhi * S, BN));
    // noisy keys whose block lies in [qlo, qhi]
    const int kfirst = qlo * S, klast = imin(L, (qhi + 1) * S) - 1;
    r.noisy0 = kfirst / BN;
    r.nnoisy = klast / BN - r.noisy0 + 1;
  } else {
    // clean key tile j is visible iff its first block <= qhi
    r.nclean = imin(nKT, cdiv((qhi + 1) * S, BN));
    r.noisy0 = 0;
    r.nnoisy = 0;
  }
  return r;
}

// Query tiles visited by key tile (kh, j): noisy query tiles
// [noisy0, noisy0 + nnoisy) then clean query tiles [clean0, clean0 + nclean).
struct QueryTileList {
  int noisy0, nnoisy, clean0, nclean;
  BD_HD int count() const { return nnoisy + nclean; }
  BD_HD void at(int t, int& qh, int& i) const {
    if (t < nnoisy) { qh = HALF_NOISY; i = noisy0 + t; }
    else { qh = HALF_CLEAN; i = clean0 + (t - nnoisy); }
  }
};

BD_HD QueryTileList query_tiles_for_key_tile(int kh, int j, int L, int S, int BM, int BN) {
  const int nQT = cdiv(L, BM);
  const int k0 = j * BN, k1 = imin(L, k0 + BN);
  const int klo = k0 / S, khi = (k1 - 1) / S;
  QueryTileList r;
  if (kh == HALF_NOISY) {
    // noisy queries whose block lies in [klo, khi]
    const int qfirst = klo * S, qlast = imin(L, (khi + 1) * S) - 1;
    r.noisy0 = qfirst / BM;
    r.nnoisy = qlast / BM - r.noisy0 + 1;
    r.clean0 = 0;
    r.nclean = 0;
  } else {
    // noisy queries with block > klo start at row (klo+1)*S
    const int qn = (klo + 1) * S;
    r.noisy0 = qn < L ? qn / BM : nQT;
    r.nnoisy = nQT - r.noisy0;
    // clean queries with block >= klo start at row klo*S
    r.clean0 = (klo * S) / BM;
    r.nclean = nQT - r.clean0;
  }
  return r;
}

// The query tiles one dK/dV workgroup visits for its key tile: tiles
// u0 + du*k, k = 0 .. K-1; each of the first K2 tiles is visited in its noisy
// and then its clean half, the others in half `rest` only, and every (tile,
// half) once per query head of the GQA group (G of them), heads innermost.
struct WalkPos;
struct QueryWalk {
  int u0, du, K, K2, rest, G;
  BD_HD int steps() const { return G * (K + K2); }
  BD_HD WalkPos first() const;
  BD_HD WalkPos last() const;
  BD_HD WalkPos at(int idx) const;  // the idx-th position (0 <= idx < steps())
};
// Position (walk tile k, half qh, query head g) in a QueryWalk.
struct WalkPos {
  int k, qh, g;
  BD_HD void next(const QueryWalk& wk) {
    if (++g < wk.G) return;
    g = 0;
    if (qh == HALF_NOISY && k < wk.K2) {
      qh = HALF_CLEAN;
      return;
    }
    ++k;
    qh = k < wk.K2 ? HALF_NOISY : wk.rest;
  }
  BD_HD int tile(const QueryWalk& wk) const { return wk.u0 + wk.du * k; }
};
BD_HD WalkPos QueryWalk::first() const { return WalkPos{0, K2 > 0 ? HALF_NOISY : rest, 0}; }
BD_HD WalkPos QueryWalk::last() const {
  return K > K2 ? WalkPos{K - 1, rest, G - 1} : WalkPos{K2 - 1, HALF_CLEAN, G - 1};
}
BD_HD WalkPos QueryWalk::at(int idx) const {
  const int n2 = 2 * G * K2;  // steps of the tiles with both halves
  if (idx < n2) {
    const int k = idx / (2 * G), r = idx - k * 2 * G;
    return r < G ? WalkPos{k, HALF_NOISY, r} : WalkPos{k, HALF_CLEAN, r - G};
  }
  const int r = idx - n2, k = K2 + r / G;
  return WalkPos{k, rest, r - (k - K2) * G};
}

// Walk of key tile (kh, j).  A clean key tile is seen by noisy query tiles
// [noisy0, nQT) and clean ones [clean0, nQT), clean0 <= noisy0; it is done by
// nsplit workgroups (split 0 .. nsplit - 1) whose walks take every nsplit-th
// tile from the top down, starting at tile nQT - 1 - split, so they have
// equal work to within one tile.  A noisy key tile is seen by noisy query
// tiles [noisy0, noisy0 + nnoisy) only and is done by one workgroup (split
// 0).  Walks start at the highest tile and move down, heads innermost, so the
// workgroups of all key tiles of one KV group read the same query tile at
// about the same time.
BD_HD QueryWalk query_walk(int kh, int j, int split, int nsplit, int L, int S, int BM, int BN, int G) {
  const QueryTileList ql = query_tiles_for_key_tile(kh, j, L, S, BM, BN);
  QueryWalk wk;
  wk.G = G;
  if (kh == HALF_CLEAN) {
    const int nQT = ql.clean0 + ql.nclean;
    wk.u0 = nQT - 1 - split;
    wk.du = -nsplit;
    wk.K = wk.u0 >= ql.clean0 ? (wk.u0 - ql.clean0) / nsplit + 1 : 0;
    wk.K2 = (ql.nnoisy > 0 && wk.u0 >= ql.noisy0) ? imin(wk.K, (wk.u0 - ql.noisy0) / nsplit + 1) : 0;
    wk.rest = HALF_CLEAN;
  } else {
    wk.u0 = ql.noisy0 + ql.nnoisy - 1;
    wk.du = -1;
    wk.K = split == 0 ? ql.nnoisy : 0;
    wk.K2 = 0;
    wk.rest = HALF_NOISY;
  }
  return wk;
}

// The first step of walk wk (query blocks of BM rows) in which no query sees
// any key of a group, steps() if there is none: every earlier block has a
// visible pair with the group.  Visibility depends on the tile and half only,
// so the scan takes one or two tests per walk tile.
BD_HD int first_unseen_step(const QueryWalk& wk, const KeyGroupSight& sight, int BM, int L) {
  for (int k = 0; k < wk.K; ++k) {
    const int q0 = (wk.u0 + wk.du * k) * BM;
    if (k < wk.K2) {
      if (!sight.sees(HALF_NOISY, q0, BM, L)) return 2 * wk.G * k;
      if (!sight.sees(HALF_CLEAN, q0, BM, L)) return 2 * wk.G * k + wk.G;
    } else if (!sight.sees(wk.rest, q0, BM, L)) {
      return 2 * wk.G * wk.K2 + wk.G * (k - wk.K2);
    }
  }
  return wk.steps();
}

}  // namespace bd
