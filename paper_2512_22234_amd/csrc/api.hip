// C-ABI entry points: argument validation, workspace layout, launch sequence.
// No exception crosses this boundary; nothing is enqueued unless every
// argument checks out.
#include <stdint.h>
#include <string.h>

#include <cmath>
#include <mutex>

#include "bd_attn.h"
#include "kernels.hpp"
#include "tiles.hpp"

// Device memory of bd_attn_bwd_noalloc: the backward's workspace (per query
// row (lse2, Delta), the float32 sums of split key-tile walks and their
// pairing counters) for callers that cannot allocate.  Every GPU that runs a
// kernel of this library holds one copy until the process ends.  In host code
// the name stands for a host-side shadow, not a device address: only the
// per-device address from hipGetSymbolAddress may be handed to kernels.
static __device__ __align__(256) char scratch[BD_ATTN_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kVersion = 100;  // 0.1.0

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct Layout {
  size_t rs = 0, part = 0, pair = 0, q = 0, k = 0, v = 0, o = 0, dout = 0, dq = 0, dk = 0, dv = 0, total = 0;
};

bool shape_ok(int B, int L, int S, int Hq, int Hkv) {
  // L <= 2^22: the kernels address one head's 2L rows of D <= 128 bf16 values
  // through 32-bit buffer offsets (2L * D * 2 bytes < 2^31)
  return B >= 1 && L >= 1 && S >= 1 && Hq >= 1 && Hkv >= 1 && Hq % Hkv == 0 && L <= (1 << 22);
}

// Rows of the Q-like and K-like arrays (per layout), times D elements each.
size_t q_rows(const bd::Shape& s) { return s.seq.cu ? (size_t)s.Hq * 2 * s.seq.T : (size_t)s.B * s.Hq * 2 * s.L; }
size_t k_rows(const bd::Shape& s) { return s.seq.cu ? (size_t)s.Hkv * 2 * s.seq.T : (size_t)s.B * s.Hkv * 2 * s.L; }

Layout make_layout(const bd::Shape& s, int dtype, bool bwd) {
  Layout w;
  const size_t nq = q_rows(s) * s.D, nk = k_rows(s) * s.D;
  size_t off = 0;
  if (bwd) {
    w.rs = off;
    off += align256(q_rows(s) * 8);
    w.part = off;
    off += align256(bd::dkdv_partial_floats(s) * 4);
    w.pair = off;
    off += align256(bd::dkdv_pair_ints(s.B, s.Hkv, s.L) * 4);
  }
  if (dtype == BD_ATTN_FP32) {
    w.q = off; off += align256(nq * 2);
    w.k = off; off += align256(nk * 2);
    w.v = off; off += align256(nk * 2);
    w.o = off; off += align256(nq * 2);
    if (bwd) {
      w.dout = off; off += align256(nq * 2);
      w.dq = off; off += align256(nq * 2);
      w.dk = off; off += align256(nk * 2);
      w.dv = off; off += align256(nk * 2);
    }
  }
  w.total = off;
  return w;
}

struct Range {
  const void* p;
  size_t n;
};

bool overlap(const Range& a, const Range& b) {
  const uintptr_t a0 = (uintptr_t)a.p, b0 = (uintptr_t)b.p;
  return a0 < b0 + b.n && b0 < a0 + a.n;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Common validation; fills the resolved shape (fixed-length layout).
int validate(int B, int L, int S, int Hq, int Hkv, int D, float scale, int dtype, bd::Shape& s) {
  if (!shape_ok(B, L, S, Hq, Hkv)) return BD_ATTN_ERR_INVALID_ARGUMENT;
  // the pairing counters of the dK/dV kernel (and its grid) are indexed with 32-bit integers
  if ((size_t)bd::DKV_PAIR_INTS * 4 * B * Hkv * bd::cdiv(L, bd::DKV_BN) > (size_t)INT32_MAX)
    return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (std::isnan(scale) || std::isinf(scale)) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (D != 64 && D != 128) return BD_ATTN_ERR_UNSUPPORTED;
  if (dtype != BD_ATTN_BF16 && dtype != BD_ATTN_FP32) return BD_ATTN_ERR_UNSUPPORTED;
  s.B = B;
  s.L = L;
  s.S = S > L ? L : S;
  s.Hq = Hq;
  s.Hkv = Hkv;
  s.D = D;
  s.G = Hq / Hkv;
  s.scale = scale > 0.f ? scale : 1.0f / std::sqrt((float)D);
  s.seq = bd::SeqLayout{nullptr, 0};
  return BD_ATTN_OK;
}

// Validation of the packed layout: n_seqs sequences, total_L tokens per copy
// in all, none longer than max_L.  The lengths themselves live in device
// memory (cu_seqlens) and are not read here.
int validate_varlen(const int32_t* cu, int n_seqs, int total_L, int max_L, int S, int Hq, int Hkv, int D,
                    float scale, int dtype, bd::Shape& s) {
  if (n_seqs < 1 || total_L < 0 || max_L < 1 || max_L > (1 << 22) || S < 1 || Hq < 1 || Hkv < 1 ||
      Hq % Hkv != 0)
    return BD_ATTN_ERR_INVALID_ARGUMENT;
  // the pairing counters of the dK/dV kernel are indexed with 32-bit integers
  if ((size_t)bd::DKV_PAIR_INTS * 4 * n_seqs * Hkv * bd::cdiv(max_L, bd::DKV_BN) > (size_t)INT32_MAX)
    return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (total_L > INT32_MAX / 2) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (cu == nullptr || !aligned(cu, 4)) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (std::isnan(scale) || std::isinf(scale)) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (D != 64 && D != 128) return BD_ATTN_ERR_UNSUPPORTED;
  if (dtype != BD_ATTN_BF16 && dtype != BD_ATTN_FP32) return BD_ATTN_ERR_UNSUPPORTED;
  s.B = n_seqs;
  s.L = max_L;
  s.S = S > max_L ? max_L : S;  // a sequence shorter than S is one block either way
  s.Hq = Hq;
  s.Hkv = Hkv;
  s.D = D;
  s.G = Hq / Hkv;
  s.scale = scale > 0.f ? scale : 1.0f / std::sqrt((float)D);
  s.seq = bd::SeqLayout{cu, total_L};
  return BD_ATTN_OK;
}

// Validation of a decode call; fills the resolved shape.
int validate_decode(int B, int S, int Hq, int Hkv, int D, int C, float scale, int dtype, bd::DecodeShape& s) {
  if (B < 1 || S < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || C < 0 || C > (1 << 22) || S > (1 << 22))
    return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (std::isnan(scale) || std::isinf(scale)) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (D != 64 && D != 128) return BD_ATTN_ERR_UNSUPPORTED;
  if (dtype != BD_ATTN_BF16) return BD_ATTN_ERR_UNSUPPORTED;
  s.B = B;
  s.S = S;
  s.Hq = Hq;
  s.Hkv = Hkv;
  s.D = D;
  s.C = C;
  s.scale = scale > 0.f ? scale : 1.0f / std::sqrt((float)D);
  // the kernels count key tiles of all items (at most every cache full) in int32
  const size_t tiles = bd::decode_items(s) * (size_t)(bd::cdiv(C, bd::DEC_KT) + bd::cdiv(S, bd::DEC_KT));
  if (tiles > (size_t)INT32_MAX / 2) return BD_ATTN_ERR_INVALID_ARGUMENT;
  return BD_ATTN_OK;
}

// Validation of the LM-head calls; fills the shape.
int validate_lce(int N, int V, int Dm, int dtype, bd::LceShape& s) {
  // buffer offsets of one 256-row operand tile stay below 2^32 bytes for
  // rows of up to 2^22 elements
  if (N < 1 || V < 1 || Dm < 256 || Dm % 256 != 0 || N > (1 << 22) || V > (1 << 22) || Dm > (1 << 16))
    return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (dtype != BD_ATTN_BF16) return BD_ATTN_ERR_UNSUPPORTED;
  s.N = N;
  s.V = V;
  s.Dm = Dm;
  return BD_ATTN_OK;
}

#define BD_TRY(expr)                                    \
  do {                                                  \
    if ((expr) != hipSuccess) return BD_ATTN_ERR_HIP;   \
  } while (0)

// Optional caller-owned events (benchmark entry points only): launch i
// records marks 2i and 2i + 1 from its own dispatch, as the kernel begins and
// as it ends, so the marks add nothing to the queue between the kernels.
struct Marks {
  hipEvent_t* ev;
  int n;
  int i = 0;
  bd::LaunchEvents next() {
    bd::LaunchEvents e;
    if (ev != nullptr && 2 * i + 1 < n) {
      e.start = ev[2 * i];
      e.stop = ev[2 * i + 1];
    }
    ++i;
    return e;
  }
};

// Device address of `scratch` on the device that runs `stream` (the current
// device for the null stream), looked up on the first call for that device
// with the device current.  Returns a status.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_for_stream(hipStream_t stream, void** out) {
  int cur = 0;
  if (hipGetDevice(&cur) != hipSuccess) return BD_ATTN_ERR_HIP;
  int dev = cur;
  if (stream != nullptr && hipStreamGetDevice(stream, &dev) != hipSuccess) return BD_ATTN_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return BD_ATTN_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    if (dev != cur && hipSetDevice(dev) != hipSuccess) return BD_ATTN_ERR_HIP;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur && hipSetDevice(cur) != hipSuccess) return BD_ATTN_ERR_HIP;
    if (e != hipSuccess || p == nullptr) return BD_ATTN_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return BD_ATTN_OK;
}

// Work of one call on a validated shape.
int fwd_impl(const bd::Shape& s, const void* Q, const void* K, const void* V, int dtype, void* O, float* LSE,
             void* ws, size_t ws_bytes, hipStream_t stream, Marks marks);
int bwd_impl(const bd::Shape& s, const void* dO, const void* Q, const void* K, const void* V, const void* O,
             const float* LSE, int dtype, void* dQ, void* dK, void* dV, void* ws, size_t ws_bytes,
             hipStream_t stream, Marks marks);

}  // namespace

extern "C" {

int bd_attn_version(void) { return kVersion; }

const char* bd_attn_status_string(int status) {
  switch (status) {
    case BD_ATTN_OK: return "ok";
    case BD_ATTN_ERR_INVALID_ARGUMENT: return "invalid argument";
    case BD_ATTN_ERR_UNSUPPORTED: return "unsupported head dimension or dtype";
    case BD_ATTN_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case BD_ATTN_ERR_HIP: return "HIP launch error";
    case BD_ATTN_ERR_EXCEEDS_SCRATCH:
      return "problem needs more workspace than the no-allocation entry point's scratch holds";
    default: return "unknown status";
  }
}

size_t bd_attn_workspace_bytes(int B, int L, int S, int Hq, int Hkv, int D, int dtype, int for_bwd) {
  bd::Shape s;
  if (validate(B, L, S, Hq, Hkv, D, 0.f, dtype, s) != BD_ATTN_OK) return 0;
  return make_layout(s, dtype, for_bwd != 0).total;
}

size_t bd_attn_varlen_workspace_bytes(int n_seqs, int total_L, int max_L, int S, int Hq, int Hkv, int D, int dtype,
                                      int for_bwd) {
  bd::Shape s;
  static const int32_t probe = 0;  // stands in for cu_seqlens: only the sizes matter here
  if (validate_varlen(&probe, n_seqs, total_L, max_L, S, Hq, Hkv, D, 0.f, dtype, s) != BD_ATTN_OK) return 0;
  return make_layout(s, dtype, for_bwd != 0).total;
}

int bd_attn_classify_tiles_host(int L, int S, int BM, int BN, int8_t* out) {
  if (L < 1 || S < 1 || BM < 1 || BN < 1 || out == nullptr) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (S > L) S = L;
  const int nqt = bd::cdiv(L, BM), nkt = bd::cdiv(L, BN);
  const int nq = 2 * nqt, nk = 2 * nkt;
  for (int a = 0; a < nq; ++a) {
    const int qh = a / nqt, i = a % nqt;
    const int q0 = i * BM, q1 = bd::imin(L, q0 + BM);
    for (int c = 0; c < nk; ++c) {
      const int kh = c / nkt, j = c % nkt;
      const int k0 = j * BN, k1 = bd::imin(L, k0 + BN);
      out[(size_t)a * nk + c] =
          (int8_t)bd::classify_pair(qh, q0, q1, kh, k0, k1, S, (q1 - q0) == BM && (k1 - k0) == BN);
    }
  }
  return BD_ATTN_OK;
}

int bd_attn_visit_lists_host(int L, int S, int BM, int BN, int by_key_tile, int nsplit, int8_t* out) {
  if (L < 1 || S < 1 || BM < 1 || BN < 1 || out == nullptr) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (by_key_tile && nsplit != 2 && nsplit != 4) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (S > L) S = L;
  const int nqt = bd::cdiv(L, BM), nkt = bd::cdiv(L, BN);
  const int nq = 2 * nqt, nk = 2 * nkt;
  memset(out, 0, (size_t)nq * nk);
  if (!by_key_tile) {
    for (int a = 0; a < nq; ++a) {
      const int qh = a / nqt, q0 = (a % nqt) * BM, q1 = bd::imin(L, q0 + BM);
      const int qA = (q0 / S) * S, qB = ((q1 - 1) / S) * S;
      const bd::FullRange fr = bd::full_range_vs_query_tile(qh, q0, q1, L, S, BM);
      const bd::KeyTileList kl = bd::key_tiles_for_query_tile(qh, a % nqt, L, S, BM, BN);
      // the forward and dQ kernels run the first t_main tiles with no visibility test
      const int t_main = bd::imin(kl.count(), fr.full_prefix(BN));
      for (int t = 0; t < kl.count(); ++t) {
        int kh, j;
        kl.at(t, kh, j);
        if (j < 0 || j >= nkt) return BD_ATTN_ERR_INVALID_ARGUMENT;
        const int k0 = j * BN, k1 = bd::imin(L, k0 + BN);
        const bool full = (q1 - q0) == BM && (k1 - k0) == BN;
        const int ref = bd::classify_pair(qh, q0, q1, kh, k0, k1, S, full);
        const int fast = bd::classify_vs_query_tile(qh, qA, qB, S, kh, k0, k1, full);
        const bool ok = fast == ref && fr.full(kh, k0, BN) == (ref == bd::TILE_FULL) &&
                        (t >= t_main || ref == bd::TILE_FULL);
        out[(size_t)a * nk + kh * nkt + j] += (int8_t)(ok ? 1 : 64);
      }
    }
  } else {
    for (int c = 0; c < nk; ++c) {
      const int kh = c / nkt, j = c % nkt, k0 = j * BN, k1 = bd::imin(L, k0 + BN);
      const int kA = (k0 / S) * S, kB = ((k1 - 1) / S) * S;
      const bd::FullRange fr = bd::full_range_vs_key_tile(kh, k0, k1, L, S, BN);
      // the walks of the workgroups that own this key tile, as the kernel
      // takes them (one query head: the kernel repeats each (tile, half)
      // once per head of the group)
      for (int split = 0; split < nsplit; ++split) {
        const bd::QueryWalk wk = bd::query_walk(kh, j, split, nsplit, L, S, BM, BN, 1);
        bd::WalkPos pos = wk.first(), prev = pos;
        for (int t = 0; t < wk.steps(); ++t, pos.next(wk)) {
          prev = pos;
          const int qh = pos.qh, i = pos.tile(wk);
          if (i < 0 || i >= nqt) return BD_ATTN_ERR_INVALID_ARGUMENT;
          const int q0 = i * BM, q1 = bd::imin(L, q0 + BM);
          const bool full = (q1 - q0) == BM && (k1 - k0) == BN;
          const int ref = bd::classify_pair(qh, q0, q1, kh, k0, k1, S, full);
          const int fast = bd::classify_vs_key_tile(kh, kA, kB, S, qh, q0, q1, full);
          const bool ok = fast == ref && fr.full(qh, q0, BM) == (ref == bd::TILE_FULL);
          out[(size_t)(qh * nqt + i) * nk + c] += (int8_t)(ok ? 1 : 64);
        }
        // the kernel repeats the last position's copy past the end of the walk
        const bd::WalkPos l = wk.last();
        if (wk.steps() > 0 && (l.k != prev.k || l.qh != prev.qh || l.g != prev.g)) return BD_ATTN_ERR_INVALID_ARGUMENT;
        // positions by index, over one and over three query heads
        for (int G = 1; G <= 3; G += 2) {
          const bd::QueryWalk wg = bd::query_walk(kh, j, split, nsplit, L, S, BM, BN, G);
          bd::WalkPos ps = wg.first();
          for (int t = 0; t < wg.steps(); ++t, ps.next(wg)) {
            const bd::WalkPos a = wg.at(t);
            if (a.k != ps.k || a.qh != ps.qh || a.g != ps.g) return BD_ATTN_ERR_INVALID_ARGUMENT;
          }
        }
        // clean key tiles: for each 32-key group, the first step of the walk
        // with no visible pair, against a scan of the pair classes
        if (kh == bd::HALF_CLEAN && BN % 32 == 0) {
          for (int g = 0; g < BN / 32; ++g) {
            const int gk0 = k0 + 32 * g, gk1 = bd::imin(k1, gk0 + 32);
            int want = wk.steps();
            bd::WalkPos ps = wk.first();
            for (int t = 0; t < wk.steps(); ++t, ps.next(wk)) {
              const int q0 = ps.tile(wk) * BM, q1 = bd::imin(L, q0 + BM);
              if (gk0 >= gk1 || bd::classify_pair(ps.qh, q0, q1, kh, gk0, gk1, S, false) == bd::TILE_EMPTY) {
                want = t;
                break;
              }
            }
            if (bd::first_unseen_step(wk, bd::KeyGroupSight(kh, gk0, k1, L, S), BM, L) != want)
              return BD_ATTN_ERR_INVALID_ARGUMENT;
          }
        }
      }
    }
  }
  return BD_ATTN_OK;
}

int bd_attn_mask_windows_host(int L, int S, int by_key, int8_t* out) {
  if (L < 1 || S < 1 || out == nullptr) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (S > L) S = L;
  const int N = 2 * L;
  memset(out, 0, (size_t)N * N);
  for (int a = 0; a < N; ++a) {  // the row's own position
    const int ah = a / L, ap = a % L, a0 = (ap / S) * S;
    for (int oh = 0; oh < 2; ++oh) {  // the other side's half
      const bd::PosWindow win = by_key ? bd::queries_seeing(ah, oh, a0, L, S, true)
                                       : bd::keys_visible_from(ah, oh, a0, L, S, true);
      for (int x = win.lo; x < win.hi; ++x) {
        const int other = oh * L + x;
        if (by_key) out[(size_t)other * N + a] = 1;  // query `other` sees key a
        else out[(size_t)a * N + other] = 1;         // query a sees key `other`
      }
    }
  }
  return BD_ATTN_OK;
}

int bd_attn_group_windows_host(int L, int S, int by_key, int group, int8_t* out) {
  if (L < 1 || S < 1 || group < 1 || out == nullptr) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (S > L) S = L;
  const int N = 2 * L;
  memset(out, 0, (size_t)N * N);
  for (int a = 0; a < N; ++a) {  // the row's own position; its run is [r0, r1) of its half
    const int ah = a / L, ap = a % L, r0 = (ap / group) * group, r1 = bd::imin(L, r0 + group);
    for (int oh = 0; oh < 2; ++oh) {
      const bd::PosWindow win = by_key ? bd::wave_queries_seeing(ah, oh, r0, r1, L, S)
                                       : bd::wave_keys_visible(ah, oh, r0, r1, L, S);
      for (int x = win.lo; x < win.hi; ++x) {
        const int other = oh * L + x;
        if (by_key) out[(size_t)other * N + a] = 1;
        else out[(size_t)a * N + other] = 1;
      }
    }
  }
  return BD_ATTN_OK;
}

int bd_attn_fwd(const void* Q, const void* K, const void* V, int B, int L, int S, int Hq, int Hkv, int D,
                float scale, int dtype, void* O, float* LSE, void* ws, size_t ws_bytes, hipStream_t stream) {
  bd::Shape s;
  const int st = validate(B, L, S, Hq, Hkv, D, scale, dtype, s);
  if (st != BD_ATTN_OK) return st;
  return fwd_impl(s, Q, K, V, dtype, O, LSE, ws, ws_bytes, stream, Marks{nullptr, 0});
}

int bd_attn_fwd_marked(const void* Q, const void* K, const void* V, int B, int L, int S, int Hq, int Hkv,
                       int D, float scale, int dtype, void* O, float* LSE, void* ws, size_t ws_bytes,
                       hipStream_t stream, hipEvent_t* marks, int n_marks) {
  bd::Shape s;
  const int st = validate(B, L, S, Hq, Hkv, D, scale, dtype, s);
  if (st != BD_ATTN_OK) return st;
  return fwd_impl(s, Q, K, V, dtype, O, LSE, ws, ws_bytes, stream, Marks{marks, n_marks});
}

int bd_attn_bwd(const void* dO, const void* Q, const void* K, const void* V, const void* O, const float* LSE,
                int B, int L, int S, int Hq, int Hkv, int D, float scale, int dtype, void* dQ, void* dK,
                void* dV, void* ws, size_t ws_bytes, hipStream_t stream) {
  bd::Shape s;
  const int st = validate(B, L, S, Hq, Hkv, D, scale, dtype, s);
  if (st != BD_ATTN_OK) return st;
  return bwd_impl(s, dO, Q, K, V, O, LSE, dtype, dQ, dK, dV, ws, ws_bytes, stream, Marks{nullptr, 0});
}

int bd_attn_bwd_marked(const void* dO, const void* Q, const void* K, const void* V, const void* O,
                       const float* LSE, int B, int L, int S, int Hq, int Hkv, int D, float scale, int dtype,
                       void* dQ, void* dK, void* dV, void* ws, size_t ws_bytes, hipStream_t stream,
                       hipEvent_t* marks, int n_marks) {
  bd::Shape s;
  const int st = validate(B, L, S, Hq, Hkv, D, scale, dtype, s);
  if (st != BD_ATTN_OK) return st;
  return bwd_impl(s, dO, Q, K, V, O, LSE, dtype, dQ, dK, dV, ws, ws_bytes, stream, Marks{marks, n_marks});
}

int bd_attn_bwd_noalloc(const void* dO, const void* Q, const void* K, const void* V, const void* O,
                        const float* LSE, int B, int L, int S, int Hq, int Hkv, int D, float scale, int dtype,
                        void* dQ, void* dK, void* dV, hipStream_t stream) {
  bd::Shape s;
  const int st = validate(B, L, S, Hq, Hkv, D, scale, dtype, s);
  if (st != BD_ATTN_OK) return st;
  if (make_layout(s, dtype, true).total > (size_t)BD_ATTN_NOALLOC_SCRATCH_BYTES) return BD_ATTN_ERR_EXCEEDS_SCRATCH;
  // the argument checks that need no workspace, before the first HIP call
  if (!dO || !Q || !K || !V || !O || !LSE || !dQ || !dK || !dV) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (!aligned(dO, 16) || !aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16) ||
      !aligned(LSE, 4) || !aligned(dQ, 16) || !aligned(dK, 16) || !aligned(dV, 16))
    return BD_ATTN_ERR_INVALID_ARGUMENT;
  void* ws = nullptr;
  const int sst = scratch_for_stream(stream, &ws);
  if (sst != BD_ATTN_OK) return sst;
  return bwd_impl(s, dO, Q, K, V, O, LSE, dtype, dQ, dK, dV, ws, (size_t)BD_ATTN_NOALLOC_SCRATCH_BYTES, stream,
                  Marks{nullptr, 0});
}

int bd_attn_varlen_fwd(const void* Q, const void* K, const void* V, const int32_t* cu_seqlens, int n_seqs,
                       int total_L, int max_L, int S, int Hq, int Hkv, int D, float scale, int dtype, void* O,
                       float* LSE, void* ws, size_t ws_bytes, hipStream_t stream) {
  bd::Shape s;
  const int st = validate_varlen(cu_seqlens, n_seqs, total_L, max_L, S, Hq, Hkv, D, scale, dtype, s);
  if (st != BD_ATTN_OK) return st;
  return fwd_impl(s, Q, K, V, dtype, O, LSE, ws, ws_bytes, stream, Marks{nullptr, 0});
}

int bd_attn_varlen_bwd(const void* dO, const void* Q, const void* K, const void* V, const void* O,
                       const float* LSE, const int32_t* cu_seqlens, int n_seqs, int total_L, int max_L, int S,
                       int Hq, int Hkv, int D, float scale, int dtype, void* dQ, void* dK, void* dV, void* ws,
                       size_t ws_bytes, hipStream_t stream) {
  bd::Shape s;
  const int st = validate_varlen(cu_seqlens, n_seqs, total_L, max_L, S, Hq, Hkv, D, scale, dtype, s);
  if (st != BD_ATTN_OK) return st;
  return bwd_impl(s, dO, Q, K, V, O, LSE, dtype, dQ, dK, dV, ws, ws_bytes, stream, Marks{nullptr, 0});
}

size_t bd_attn_decode_workspace_bytes(int B, int S, int Hq, int Hkv, int D, int capacity, int dtype) {
  bd::DecodeShape s;
  if (validate_decode(B, S, Hq, Hkv, D, capacity, 0.f, dtype, s) != BD_ATTN_OK) return 0;
  return bd::decode_workspace_bytes(s);
}

int bd_attn_decode_fwd(const void* Q, const void* K_cache, const void* V_cache, const void* K_new,
                       const void* V_new, const int32_t* cache_lens, int B, int S, int Hq, int Hkv, int D,
                       int capacity, float scale, int dtype, void* O, float* LSE, void* ws, size_t ws_bytes,
                       hipStream_t stream) {
  bd::DecodeShape s;
  const int st = validate_decode(B, S, Hq, Hkv, D, capacity, scale, dtype, s);
  if (st != BD_ATTN_OK) return st;
  const size_t need = bd::decode_workspace_bytes(s);
  const bool cache = capacity > 0;
  if (!Q || !K_new || !V_new || !cache_lens || !O || !LSE || !ws || (cache && (!K_cache || !V_cache)))
    return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (!aligned(Q, 16) || !aligned(K_new, 16) || !aligned(V_new, 16) || !aligned(K_cache, 16) ||
      !aligned(V_cache, 16) || !aligned(cache_lens, 4) || !aligned(O, 16) || !aligned(LSE, 4) || !aligned(ws, 16))
    return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (ws_bytes < need) return BD_ATTN_ERR_WORKSPACE_TOO_SMALL;
  const size_t nq = (size_t)B * Hq * S, nkn = (size_t)B * Hkv * S * D, nkc = (size_t)B * Hkv * capacity * D;
  const Range in[] = {{Q, nq * D * 2}, {K_new, nkn * 2}, {V_new, nkn * 2}, {K_cache, nkc * 2},
                      {V_cache, nkc * 2}, {cache_lens, (size_t)B * 4}};
  const Range out[] = {{O, nq * D * 2}, {LSE, nq * 4}, {ws, need}};
  for (const Range& o : out)
    for (const Range& i : in)
      if (i.p && overlap(o, i)) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (overlap(out[0], out[1]) || overlap(out[0], out[2]) || overlap(out[1], out[2]))
    return BD_ATTN_ERR_INVALID_ARGUMENT;
  (void)hipGetLastError();
  return bd::launch_decode(s, Q, K_cache, V_cache, K_new, V_new, cache_lens, O, LSE, ws, stream) == hipSuccess
             ? BD_ATTN_OK
             : BD_ATTN_ERR_HIP;
}

size_t bd_lce_workspace_bytes(int N, int V, int Dm, int dtype, int for_bwd) {
  bd::LceShape s;
  if (validate_lce(N, V, Dm, dtype, s) != BD_ATTN_OK) return 0;
  return for_bwd ? bd::lce_bwd_workspace_bytes(s) : bd::lce_fwd_workspace_bytes(s);
}

size_t bd_lce_logits_bytes(int N, int V, int Dm, int dtype) {
  bd::LceShape s;
  if (validate_lce(N, V, Dm, dtype, s) != BD_ATTN_OK) return 0;
  return bd::lce_logits_bytes(s);
}

int bd_lce_fwd(const void* H, const void* W, const int32_t* targets, int N, int V, int Dm, int dtype, float* lse,
               float* logp, float* logits, void* ws, size_t ws_bytes, hipStream_t stream) {
  bd::LceShape s;
  const int st = validate_lce(N, V, Dm, dtype, s);
  if (st != BD_ATTN_OK) return st;
  if (!H || !W || !targets || !lse || !logp || !ws) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (!aligned(H, 16) || !aligned(W, 16) || !aligned(targets, 4) || !aligned(lse, 4) || !aligned(logp, 4) ||
      !aligned(logits, 16) || !aligned(ws, 16))
    return BD_ATTN_ERR_INVALID_ARGUMENT;
  const size_t need = bd::lce_fwd_workspace_bytes(s);
  if (ws_bytes < need) return BD_ATTN_ERR_WORKSPACE_TOO_SMALL;
  const Range in[] = {{H, (size_t)N * Dm * 2}, {W, (size_t)V * Dm * 2}, {targets, (size_t)N * 4}};
  const Range out[] = {{lse, (size_t)N * 4}, {logp, (size_t)N * 4}, {ws, need},
                       {logits, logits ? bd::lce_logits_bytes(s) : 0}};
  for (const Range& o : out)
    for (const Range& i : in)
      if (o.p && overlap(o, i)) return BD_ATTN_ERR_INVALID_ARGUMENT;
  for (int a = 0; a < 4; ++a)
    for (int c = a + 1; c < 4; ++c)
      if (out[a].p && out[c].p && overlap(out[a], out[c])) return BD_ATTN_ERR_INVALID_ARGUMENT;
  (void)hipGetLastError();
  return bd::launch_lce_fwd(s, H, W, targets, lse, logp, logits, ws, stream) == hipSuccess ? BD_ATTN_OK
                                                                                          : BD_ATTN_ERR_HIP;
}

int bd_lce_bwd(const void* H, const void* W, const int32_t* targets, const float* lse, const float* dlogp,
               const float* logits, int N, int V, int Dm, int dtype, void* dH, void* dW, void* ws, size_t ws_bytes,
               hipStream_t stream) {
  bd::LceShape s;
  const int st = validate_lce(N, V, Dm, dtype, s);
  if (st != BD_ATTN_OK) return st;
  if (!H || !W || !targets || !lse || !dlogp || !dH || !dW || !ws) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (!aligned(H, 16) || !aligned(W, 16) || !aligned(targets, 4) || !aligned(lse, 4) || !aligned(dlogp, 4) ||
      !aligned(dH, 16) || !aligned(dW, 16) || !aligned(ws, 16) || !aligned(logits, 16))
    return BD_ATTN_ERR_INVALID_ARGUMENT;
  const size_t need = bd::lce_bwd_workspace_bytes(s);
  if (ws_bytes < need) return BD_ATTN_ERR_WORKSPACE_TOO_SMALL;
  const Range in[] = {{H, (size_t)N * Dm * 2}, {W, (size_t)V * Dm * 2}, {targets, (size_t)N * 4},
                      {lse, (size_t)N * 4}, {dlogp, (size_t)N * 4}, {logits, logits ? bd::lce_logits_bytes(s) : 0}};
  const Range out[] = {{dH, (size_t)N * Dm * 2}, {dW, (size_t)V * Dm * 2}, {ws, need}};
  for (const Range& o : out)
    for (const Range& i : in)
      if (overlap(o, i)) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (overlap(out[0], out[1]) || overlap(out[0], out[2]) || overlap(out[1], out[2])) return BD_ATTN_ERR_INVALID_ARGUMENT;
  (void)hipGetLastError();
  return bd::launch_lce_bwd(s, H, W, targets, lse, dlogp, logits, dH, dW, ws, stream) == hipSuccess
             ? BD_ATTN_OK
             : BD_ATTN_ERR_HIP;
}

int bd_lce_objective(const float* logp, const float* logp_old, const float* logp_ref, const float* adv,
                     const float* weight, int N, int kind, float eps, float beta, float* loss, float* dlogp,
                     hipStream_t stream) {
  if (N < 1 || (kind != BD_LCE_CE && kind != BD_LCE_DIPO)) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (std::isnan(eps) || std::isinf(eps) || eps < 0.f || std::isnan(beta) || std::isinf(beta) || beta < 0.f)
    return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (!logp || !weight || !loss || !dlogp) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (kind == BD_LCE_DIPO && (!logp_old || !adv || (beta != 0.f && !logp_ref))) return BD_ATTN_ERR_INVALID_ARGUMENT;
  const float* ptrs[] = {logp, logp_old, logp_ref, adv, weight, loss, dlogp};
  for (const float* q : ptrs)
    if (!aligned(q, 4)) return BD_ATTN_ERR_INVALID_ARGUMENT;
  const size_t nb = (size_t)N * 4;
  const Range in[] = {{logp, nb}, {logp_old, logp_old ? nb : 0}, {logp_ref, logp_ref ? nb : 0},
                      {adv, adv ? nb : 0}, {weight, nb}};
  const Range out[] = {{loss, nb}, {dlogp, nb}};
  for (const Range& o : out)
    for (const Range& i : in)
      if (i.p && overlap(o, i)) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (overlap(out[0], out[1])) return BD_ATTN_ERR_INVALID_ARGUMENT;
  (void)hipGetLastError();
  return bd::launch_lce_objective(N, kind, eps, beta, logp, logp_old, logp_ref, adv, weight, loss, dlogp, stream) ==
                 hipSuccess
             ? BD_ATTN_OK
             : BD_ATTN_ERR_HIP;
}

const char* bd_attn_stage_names(int for_bwd, int dtype) {
  if (dtype == BD_ATTN_FP32)
    return for_bwd ? "cast_q,cast_k,cast_v,cast_o,cast_do,bwd_dq,bwd_dkdv,cast_dq,cast_dk,cast_dv"
                   : "cast_q,cast_k,cast_v,fwd,cast_o";
  return for_bwd ? "bwd_dq,bwd_dkdv" : "fwd";
}

}  // extern "C"

namespace {

int fwd_impl(const bd::Shape& s, const void* Q, const void* K, const void* V, int dtype, void* O, float* LSE,
             void* ws, size_t ws_bytes, hipStream_t stream, Marks marks) {
  const Layout w = make_layout(s, dtype, false);
  if (q_rows(s) == 0) return BD_ATTN_OK;  // packed layout with no tokens: nothing to read or write
  if (!Q || !K || !V || !O || !LSE || (w.total > 0 && !ws)) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16) || !aligned(LSE, 4) ||
      !aligned(ws, 16))
    return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (ws_bytes < w.total) return BD_ATTN_ERR_WORKSPACE_TOO_SMALL;
  const size_t esz = dtype == BD_ATTN_FP32 ? 4 : 2;
  const size_t nq = q_rows(s) * s.D, nk = k_rows(s) * s.D;
  const Range in[] = {{Q, nq * esz}, {K, nk * esz}, {V, nk * esz}};
  const Range out[] = {{O, nq * esz}, {LSE, q_rows(s) * 4}, {ws, w.total}};
  for (const Range& o : out)
    for (const Range& i : in)
      if (overlap(o, i)) return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (overlap(out[0], out[1]) || overlap(out[0], out[2]) || overlap(out[1], out[2]))
    return BD_ATTN_ERR_INVALID_ARGUMENT;

  (void)hipGetLastError();  // clear a stale error so it is not reported as ours
  char* wb = static_cast<char*>(ws);
  const void *q = Q, *k = K, *v = V;
  void* o = O;
  if (dtype == BD_ATTN_FP32) {
    BD_TRY(bd::launch_cast_f32_to_bf16(static_cast<const float*>(Q), wb + w.q, nq, stream, marks.next()));
    BD_TRY(bd::launch_cast_f32_to_bf16(static_cast<const float*>(K), wb + w.k, nk, stream, marks.next()));
    BD_TRY(bd::launch_cast_f32_to_bf16(static_cast<const float*>(V), wb + w.v, nk, stream, marks.next()));
    q = wb + w.q;
    k = wb + w.k;
    v = wb + w.v;
    o = wb + w.o;
  }
  BD_TRY(bd::launch_fwd(s, q, k, v, o, LSE, stream, marks.next()));
  if (dtype == BD_ATTN_FP32) BD_TRY(bd::launch_cast_bf16_to_f32(o, static_cast<float*>(O), nq, stream, marks.next()));
  return BD_ATTN_OK;
}

int bwd_impl(const bd::Shape& s, const void* dO, const void* Q, const void* K, const void* V, const void* O,
             const float* LSE, int dtype, void* dQ, void* dK, void* dV, void* ws, size_t ws_bytes,
             hipStream_t stream, Marks marks) {
  const Layout w = make_layout(s, dtype, true);
  if (q_rows(s) == 0) return BD_ATTN_OK;  // packed layout with no tokens: nothing to read or write
  if (!dO || !Q || !K || !V || !O || !LSE || !dQ || !dK || !dV || (w.total > 0 && !ws))
    return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (!aligned(dO, 16) || !aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16) ||
      !aligned(LSE, 4) || !aligned(dQ, 16) || !aligned(dK, 16) || !aligned(dV, 16) || !aligned(ws, 16))
    return BD_ATTN_ERR_INVALID_ARGUMENT;
  if (ws_bytes < w.total) return BD_ATTN_ERR_WORKSPACE_TOO_SMALL;
  const size_t esz = dtype == BD_ATTN_FP32 ? 4 : 2;
  const size_t nq = q_rows(s) * s.D, nk = k_rows(s) * s.D;
  const Range in[] = {{dO, nq * esz}, {Q, nq * esz}, {K, nk * esz}, {V, nk * esz}, {O, nq * esz},
                      {LSE, q_rows(s) * 4}};
  const Range out[] = {{dQ, nq * esz}, {dK, nk * esz}, {dV, nk * esz}, {ws, w.total}};
  for (const Range& o : out)
    for (const Range& i : in)
      if (overlap(o, i)) return BD_ATTN_ERR_INVALID_ARGUMENT;
  for (int a = 0; a < 4; ++a)
    for (int c = a + 1; c < 4; ++c)
      if (overlap(out[a], out[c])) return BD_ATTN_ERR_INVALID_ARGUMENT;

  (void)hipGetLastError();
  char* wb = static_cast<char*>(ws);
  const void *q = Q, *k = K, *v = V, *o = O, *g = dO;
  void *dq = dQ, *dk = dK, *dv = dV;
  if (dtype == BD_ATTN_FP32) {
    BD_TRY(bd::launch_cast_f32_to_bf16(static_cast<const float*>(Q), wb + w.q, nq, stream, marks.next()));
    BD_TRY(bd::launch_cast_f32_to_bf16(static_cast<const float*>(K), wb + w.k, nk, stream, marks.next()));
    BD_TRY(bd::launch_cast_f32_to_bf16(static_cast<const float*>(V), wb + w.v, nk, stream, marks.next()));
    BD_TRY(bd::launch_cast_f32_to_bf16(static_cast<const float*>(O), wb + w.o, nq, stream, marks.next()));
    BD_TRY(bd::launch_cast_f32_to_bf16(static_cast<const float*>(dO), wb + w.dout, nq, stream, marks.next()));
    q = wb + w.q;
    k = wb + w.k;
    v = wb + w.v;
    o = wb + w.o;
    g = wb + w.dout;
    dq = wb + w.dq;
    dk = wb + w.dk;
    dv = wb + w.dv;
  }
  float* rs = reinterpret_cast<float*>(wb + w.rs);
  float* part = reinterpret_cast<float*>(wb + w.part);
  int* pair = reinterpret_cast<int*>(wb + w.pair);
  BD_TRY(bd::launch_bwd_dq(s, q, k, v, g, o, LSE, rs, pair, dq, stream, marks.next()));
  BD_TRY(bd::launch_bwd_dkdv(s, q, k, v, g, rs, dk, dv, part, pair, stream, marks.next()));
  if (dtype == BD_ATTN_FP32) {
    BD_TRY(bd::launch_cast_bf16_to_f32(dq, static_cast<float*>(dQ), nq, stream, marks.next()));
    BD_TRY(bd::launch_cast_bf16_to_f32(dk, static_cast<float*>(dK), nk, stream, marks.next()));
    BD_TRY(bd::launch_cast_bf16_to_f32(dv, static_cast<float*>(dV), nk, stream, marks.next()));
  }
  return BD_ATTN_OK;
}

}  // namespace
