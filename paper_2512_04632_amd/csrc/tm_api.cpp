// C ABI of the Turbo-Muon orthogonalizer: argument validation, per-stream
// workspace cache and the launch plan of Algorithms 1 and 2 (one launch per
// phase over the tiles of every matrix of the call).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <array>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "tm_internal.h"
#include "turbomuon.h"

namespace tmk {
hipError_t launch_elementwise_bf16(int kind, const Phase& P, hipStream_t st);
hipError_t launch_fast_bf16(int kind, int cfg, int step, const Phase& P, hipStream_t st);
hipError_t launch_phase_f32(int kind, int cfg, const Phase& P, hipStream_t st);
hipError_t launch_opt(int apply, const OptPhase& P, hipStream_t st);
hipError_t launch_small_bf16(int F, int big, const SmallPhase& P, hipStream_t st);
}  // namespace tmk

namespace {

using tmk::Entry;
using tmk::Phase;

thread_local std::string g_last_error;

tm_status fail(tm_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

// Default coefficients: the constant quintic triple, used for every iteration.
constexpr float kA = 3.4445f, kB = -4.7750f, kC = 2.0315f;

struct Workspace {
  void* ptr = nullptr;
  size_t bytes = 0;
  bool captured = false;   // used by a call under graph capture: never freed or reused in place
};

std::mutex g_mu;
using WsCache = std::map<std::pair<int, hipStream_t>, Workspace>;
WsCache g_ws;     // iteration workspace of every call
WsCache g_ws_u;   // bf16 update matrices of the optimizer step
std::map<int, bool> g_dev_ok;
// Workspaces replaced while a captured graph may still hold their address:
// freed only by tm_release_workspaces.
std::vector<void*> g_retired;

// Timing hooks: event pairs bracketing each launch while enabled.
struct TimedLaunch {
  int kind;
  hipEvent_t start, stop;
};
bool g_timing = false;
std::vector<TimedLaunch> g_timed;
static_assert(int(tmk::kNumKinds) == TM_NUM_PHASES, "one timing phase per kernel kind");
static_assert(tmk::kMaxIters == TM_MAX_ITERS, "the fused kernel's descriptor holds every iteration");
double g_time_ms[TM_NUM_PHASES];
int64_t g_time_n[TM_NUM_PHASES];

void collect_timing() {
  for (TimedLaunch& t : g_timed) {
    float ms = 0.f;
    if (hipEventSynchronize(t.stop) == hipSuccess &&
        hipEventElapsedTime(&ms, t.start, t.stop) == hipSuccess) {
      g_time_ms[t.kind] += double(ms);
      g_time_n[t.kind] += 1;
    }
    (void)hipEventDestroy(t.start);
    (void)hipEventDestroy(t.stop);
  }
  g_timed.clear();
}

// One matrix (or a batch of equal matrices stored back to back).
struct Item {
  char* x;
  uint32_t k, N;
  uint32_t kp, Np;     // padded workspace dims (set by the planner)
  uint32_t count;
  bool tall;
  bool direct;         // bf16: iteration 1 reads the caller's matrix in place of a padded copy
};

// Which items a launch covers (the others get no blocks).
enum Cover { kCoverAll, kCoverTall, kCoverCopied };

tm_status check_device(int* dev) {
  hipError_t e = hipGetDevice(dev);
  if (e != hipSuccess) return fail(TM_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  auto it = g_dev_ok.find(*dev);
  if (it == g_dev_ok.end()) {
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, *dev);
    if (e != hipSuccess)
      return fail(TM_ERR_HIP, std::string("hipGetDeviceProperties: ") + hipGetErrorString(e));
    const bool ok = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
    it = g_dev_ok.emplace(*dev, ok).first;
  }
  if (!it->second) return fail(TM_ERR_UNSUPPORTED, "device is not gfx950 (MI355X)");
  return TM_OK;
}

// Grow the (device, stream) buffer of a cache to at least `bytes`.  Under
// graph capture nothing may be allocated, freed or synchronised: the buffer
// must already be large enough, and it is then marked as captured.  A captured
// buffer keeps its address for the graphs that hold it: a later, larger eager
// call on that stream handle gets a new buffer, and the old one is retired
// (freed by tm_release_workspaces only).
tm_status get_workspace(int dev, hipStream_t st, size_t bytes, char** out, WsCache& cache = g_ws) {
  Workspace& w = cache[{dev, st}];
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(st, &cap) != hipSuccess) {
    (void)hipGetLastError();
    cap = hipStreamCaptureStatusNone;
  }
  if (cap != hipStreamCaptureStatusNone) {
    if (w.bytes < bytes)
      return fail(TM_ERR_UNSUPPORTED,
                  "the stream's workspace holds " + std::to_string(w.bytes) + " bytes, the call "
                  "needs " + std::to_string(bytes) + "; nothing can be allocated under graph "
                  "capture (make one call of this size on the stream before capturing)");
    w.captured = true;
    *out = static_cast<char*>(w.ptr);
    return TM_OK;
  }
  if (w.bytes < bytes) {
    if (w.ptr && w.captured) {
      g_retired.push_back(w.ptr);
      w.ptr = nullptr;
      w.bytes = 0;
      w.captured = false;
    } else if (w.ptr) {
      hipError_t e = hipStreamSynchronize(st);
      if (e != hipSuccess)
        return fail(TM_ERR_HIP, std::string("hipStreamSynchronize: ") + hipGetErrorString(e));
      (void)hipFree(w.ptr);
      w.ptr = nullptr;
      w.bytes = 0;
    }
    void* p = nullptr;
    if (std::getenv("TM_TEST_FAIL_ALLOC") != nullptr ||
        hipMalloc(&p, bytes) != hipSuccess || p == nullptr) {
      (void)hipGetLastError();
      return fail(TM_ERR_NO_MEMORY, "workspace allocation of " + std::to_string(bytes) +
                                        " bytes failed");
    }
    w.ptr = p;
    w.bytes = bytes;
  }
  *out = static_cast<char*>(w.ptr);
  return TM_OK;
}

uint64_t item_ws(const Item& it, int esz) {
  return tmk::ws_layout(it.kp, it.Np, uint32_t(esz)).total * it.count;
}

// Generic (fp32) path: pick per phase the largest tile whose launch still
// spans one wave of the chip's 256 compute units; otherwise the smallest.
int choose_cfg(int kind, const std::vector<Item>& items) {
  for (int cfg = 0; cfg < tmk::kNumCfg - 1; ++cfg) {
    uint64_t tiles = 0;
    for (const Item& it : items)
      tiles += uint64_t(it.count) * tmk::blocks_per_matrix(kind, cfg, it.k, it.N, it.kp, it.Np);
    if (tiles >= 256) return cfg;
  }
  return tmk::kNumCfg - 1;
}

// bf16 path: the layout tile of the call (the Gram and polynomial may run
// smaller tiles of it).  Take the largest tile whose zero padding adds at most
// 30% to the call's products and whose update still has about two waves of
// tiles for the 256 compute units; the 256 tile also needs update tiles with
// a mean K of at least 512, below which its fixed costs per tile (pipeline
// fill, the 128 KB epilogue) outweigh its faster main loop.
int choose_tile_cfg(const std::vector<Item>& items) {
  double real = 0.0;
  for (const Item& it : items)
    real += double(it.count) * (3.0 * it.k * double(it.k) * it.N + double(it.k) * it.k * it.k);
  for (int cfg = 0; cfg < tmk::kNumCfg - 1; ++cfg) {
    const uint32_t T = uint32_t(tmk::cfg_tile(cfg));
    double padded = 0.0, tiles = 0.0, ksum = 0.0;
    for (const Item& it : items) {
      uint32_t kp, Np;
      tmk::tiled_dims(it.k, it.N, T, &kp, &Np);
      padded += double(it.count) * (3.0 * kp * double(kp) * Np + double(kp) * kp * kp);
      const double t = double(it.count) * (kp / T) * (Np / T);
      tiles += t;
      ksum += t * kp;
    }
    const bool long_k = T < 256 || ksum >= 512.0 * tiles;
    if (padded <= 1.3 * real && tiles >= 480.0 && long_k) return cfg;
  }
  return tmk::kNumCfg - 1;
}

// bf16 Gram and polynomial phases: the layout tile T (kp, Np multiples of
// it) is halved, down to 64 (or 32 with `small`: one-wave tiles, not for the
// first Gram, whose row partials cover 64 columns), until the phase has one
// and a half waves of tiles for the 256 compute units, or one wave at least
// three quarters full (a tile per compute unit: no second, partly filled
// wave); these phases have about k^2 / T^2 / 2 tiles per matrix against
// k N / T^2 for the update.  (The 72 matrices of a 12-layer 768-wide model:
// 432 tiles of 256 beat 1512 of 128 by 7% per call.)
int choose_sym_cfg(int kind, int tcfg, const std::vector<Item>& items, bool small = false) {
  int cfg = tcfg;
  const int last = small ? tmk::kCfgSym32 : tmk::kNumCfg - 1;
  while (cfg < last) {
    uint64_t tiles = 0;
    for (const Item& it : items)
      tiles += uint64_t(it.count) * tmk::blocks_per_matrix(kind, cfg, it.k, it.N, it.kp, it.Np);
    if (tiles >= 384 || (tiles >= 192 && tiles <= 256)) break;
    ++cfg;
  }
  return cfg;
}

struct Plan {
  const std::vector<Item>* items;
  std::vector<uint64_t> ws_off;   // byte offset of each item's workspace region
  char* ws;
  int esz;
  hipStream_t st;
  int tcfg = 0;                   // bf16: the call's layout tile
  bool timed = true;              // the timing hooks may bracket this call's launches
};

// bf16 update of one launch of a call split over several launches: the
// largest tile (at most the layout tile) with about two waves of tiles.
int choose_update_cfg(int tcfg, const std::vector<Item>& items) {
  for (int cfg = tcfg; cfg < tmk::kNumCfg - 1; ++cfg) {
    uint64_t tiles = 0;
    for (const Item& it : items)
      tiles += uint64_t(it.count) * tmk::blocks_per_matrix(tmk::kKindUpdate, cfg, it.k, it.N, it.kp, it.Np);
    if (tiles >= 480) return cfg;
  }
  return tmk::kNumCfg - 1;
}

// Compute units of the MI355X: the blocks of one full wave of the large tiles.
constexpr int kWave = 256;

// K step (elements per ring stage) of a 4-wave or one-wave bf16 launch.  A
// 96 KB ring (128 for the 64 tile, 64 for the 128 tile) holds one block per
// compute unit, so it serves launches of at most one wave of blocks; a 48 KB
// ring (64 for the 64 tile, 128 for the 32 tile) holds three, which suits a
// launch of any size; else 32 (the 128 tile's many-block launches).  Every K
// of the launch must be a multiple of the step: the Gram contracts over Np,
// the polynomial and the update over kp.  (The 256 tile's ring is fixed.)
int k_step(int kind, int cfg, const Phase& P) {
  const int T = tmk::cfg_tile(cfg);
  int step = 32;
  if (T == 128 && P.total <= kWave) step = 64;
  if (T == 64) step = P.total <= kWave ? 128 : 64;
  if (T == 32) step = 128;
  for (int e = 0; e < P.nent && step > 32; ++e) {
    const uint32_t K = kind == tmk::kKindGram ? P.e[e].Np : P.e[e].kp;
    if (P.e[e].tiles_per != 0u && K % uint32_t(step) != 0u) step = 32;
  }
  return step;
}

// Enqueue one kernel launch of a prepared phase descriptor (timed when the
// timing hooks are on).
tm_status fire(const Plan& pl, int kind, int cfg, const Phase& P) {
  TimedLaunch tl{kind, nullptr, nullptr};
  if (g_timing && pl.timed && P.total > 0) {
    if (hipEventCreate(&tl.start) != hipSuccess || hipEventCreate(&tl.stop) != hipSuccess)
      return fail(TM_ERR_HIP, "hipEventCreate failed");
    (void)hipEventRecord(tl.start, pl.st);
  }
  hipError_t e;
  if (pl.esz == 4)
    e = tmk::launch_phase_f32(kind, cfg, P, pl.st);
  else if (kind == tmk::kKindFrob || kind == tmk::kKindAolVector || kind == tmk::kKindApplyScale)
    e = tmk::launch_elementwise_bf16(kind, P, pl.st);
  else
    e = tmk::launch_fast_bf16(kind, cfg, k_step(kind, cfg, P), P, pl.st);
  if (tl.start) {
    (void)hipEventRecord(tl.stop, pl.st);
    g_timed.push_back(tl);
  }
  if (e != hipSuccess) return fail(TM_ERR_HIP, std::string("kernel launch: ") + hipGetErrorString(e));
  return TM_OK;
}

// Entries of one launch: a run of positions [first, first + n) of the launch
// order.  A run of n > 1 single matrices of one shape whose workspace regions
// follow each other is one kPtrTab entry; otherwise n = 1.
struct Run {
  size_t first, n;
};

// One launch of `kind` per chunk of at most kMaxEntries entries and kMaxPtrs
// table pointers.
tm_status launch(const Plan& pl, int kind, int cfg, int src, int dst, float a, float b, float c,
                 uint32_t flags, int aux, Cover cover = kCoverAll) {
  const std::vector<Item>& items = *pl.items;
  // update launches take their largest products first (the longest tiles
  // start first); every entry carries its own workspace offset
  std::vector<size_t> idx(items.size());
  for (size_t i = 0; i < idx.size(); ++i) idx[i] = i;
  if (kind == tmk::kKindUpdate)
    std::stable_sort(idx.begin(), idx.end(), [&](size_t x, size_t y) {
      const Item& u = items[x];
      const Item& v = items[y];
      return double(u.k) * u.k * u.N * u.count > double(v.k) * v.k * v.N * v.count;
    });
  auto joins = [&](size_t prev, size_t next) {
    const Item& u = items[idx[prev]];
    const Item& v = items[idx[next]];
    return u.count == 1u && v.count == 1u && u.k == v.k && u.N == v.N && u.kp == v.kp &&
           u.Np == v.Np && u.tall == v.tall && u.direct == v.direct &&
           pl.ws_off[idx[next]] == pl.ws_off[idx[prev]] + item_ws(u, pl.esz);
  };
  std::vector<std::vector<Run>> chunks(1);
  int ptrs = 0;
  for (size_t i = 0; i < idx.size(); ++i) {
    std::vector<Run>& ch = chunks.back();
    if (!ch.empty() && joins(i - 1, i)) {
      Run& r = ch.back();
      const int need = r.n == 1 ? 2 : 1;   // a run of two starts the table
      if (ptrs + need <= tmk::kMaxPtrs) {
        ++r.n;
        ptrs += need;
        continue;
      }
    }
    if (ch.size() == size_t(tmk::kMaxEntries) || ptrs == tmk::kMaxPtrs) {
      chunks.emplace_back();
      ptrs = 0;
    }
    chunks.back().push_back(Run{i, 1});
  }
  for (const std::vector<Run>& ch : chunks) {
    Phase P;
    std::memset(&P, 0, sizeof(P));
    // a call split over several launches picks each launch's tile for that
    // launch's matrices (the last one may be much smaller); a product's
    // arithmetic does not depend on the tile size
    int ccfg = cfg;
    if (pl.esz == 2 && chunks.size() > 1 &&
        (kind == tmk::kKindGram || kind == tmk::kKindPoly || kind == tmk::kKindUpdate)) {
      std::vector<Item> chunk;
      for (const Run& r : ch)
        for (size_t i = r.first; i < r.first + r.n; ++i) chunk.push_back(items[idx[i]]);
      ccfg = kind == tmk::kKindUpdate
                 ? choose_update_cfg(pl.tcfg, chunk)
                 : choose_sym_cfg(kind, pl.tcfg, chunk, kind == tmk::kKindPoly || flags == 0u);
    }
    uint64_t start = 0;
    uint32_t xp = 0;
    const size_t n = ch.size();
    for (size_t e = 0; e < n; ++e) {
      const Run& r = ch[e];
      const Item& it = items[idx[r.first]];
      Entry& E = P.e[e];
      E.x = it.x;
      E.ws256 = uint32_t(pl.ws_off[idx[r.first]] >> 8);
      E.k = it.k;
      E.N = it.N;
      E.kp = it.kp;
      E.Np = it.Np;
      E.count = r.n > 1 ? uint32_t(r.n) : it.count;
      E.flags = (it.tall ? tmk::kTall : 0u) | (it.direct ? tmk::kDirect : 0u);
      if (r.n > 1) {
        E.flags |= tmk::kPtrTab;
        E.xbase = xp;
        for (size_t i = r.first; i < r.first + r.n; ++i) P.xp[xp++] = items[idx[i]].x;
      }
      E.tile_start = uint32_t(start);
      const bool skip = (cover == kCoverTall && !it.tall) || (cover == kCoverCopied && it.direct);
      E.tiles_per = skip ? 0u : tmk::blocks_per_matrix(kind, ccfg, it.k, it.N, it.kp, it.Np);
      start += uint64_t(E.tiles_per) * E.count;
    }
    if (start >= (uint64_t(1) << 31))
      return fail(TM_ERR_UNSUPPORTED, "too many tiles in one launch");
    P.nent = int32_t(n);
    P.total = int32_t(start);
    P.ws = pl.ws;
    P.src = src;
    P.dst = dst;
    P.a = a;
    P.b = b;
    P.c = c;
    P.flags = flags;
    P.aux = aux;
    P.tail_base = 0;
    tm_status s = TM_OK;
    // A bf16 matrix-core launch whose entries' tiles differ in K deals whole
    // matrices round-robin to the XCDs (kByMatrix) when that splits the work
    // evenly (every XCD within 10% of an eighth, the cost of a tile taken as
    // its K): the default chunks of consecutive tiles per XCD would give the
    // first XCDs all the long tiles of a largest-first launch.  A launch of a
    // few matrices keeps the chunks.
    const bool mc0 = kind == tmk::kKindGram || kind == tmk::kKindPoly || kind == tmk::kKindUpdate;
    bool by_matrix = false;
    if (pl.esz == 2 && mc0) {
      uint32_t kmin = UINT32_MAX, kmax = 0;
      for (int e = 0; e < P.nent; ++e) {
        if (P.e[e].tiles_per == 0u) continue;
        const uint32_t K = kind == tmk::kKindGram ? P.e[e].Np : P.e[e].kp;
        kmin = std::min(kmin, K);
        kmax = std::max(kmax, K);
      }
      if (kmin != kmax) {
        uint64_t q[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        double cost[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        uint64_t g0 = 0;
        for (int e = 0; e < P.nent; ++e) {
          const uint64_t c = P.e[e].count;
          const double K = kind == tmk::kKindGram ? P.e[e].Np : P.e[e].kp;
          for (int x = 0; x < 8; ++x) {
            const uint64_t i0 = uint64_t((x - int(g0 & 7u) + 8) & 7);
            const uint64_t t = (i0 < c ? (c - 1 - i0) / 8 + 1 : 0) * P.e[e].tiles_per;
            q[x] += t;
            cost[x] += double(t) * K;
          }
          g0 += c;
        }
        double sum = 0.0, top = 0.0;
        for (int x = 0; x < 8; ++x) {
          sum += cost[x];
          top = std::max(top, cost[x]);
        }
        if (top <= 1.1 * sum / 8.0) {
          P.flags |= tmk::kByMatrix;
          P.total = int32_t(8 * *std::max_element(q, q + 8));
          by_matrix = true;
        }
      }
    }
    // bf16 matrix-core phases on 256 x 256 tiles whose last wave would be at
    // most a quarter full: the full waves run as usual, the remaining tiles as
    // 2 x 2 sub-tiles of 128 x 128 in a second launch that fits in one wave
    // (same per-element arithmetic, four times the blocks for the idle units);
    // an update tail of at most 16 tiles as 4 x 4 sub-tiles of 64 x 64.
    const bool mc = kind == tmk::kKindGram || kind == tmk::kKindPoly || kind == tmk::kKindUpdate;
    const int tail = (!by_matrix && pl.esz == 2 && ccfg == 0 && mc && P.total > kWave && P.total % kWave <= kWave / 4)
                         ? P.total % kWave
                         : 0;
    if (tail > 0) {
      P.total -= tail;
      s = fire(pl, kind, ccfg, P);
      Phase Q = P;
      const bool f4 = kind == tmk::kKindUpdate && 16 * tail <= kWave;
      Q.flags |= tmk::kTail | (f4 ? tmk::kTail4 : 0u);
      Q.tail_base = P.total;
      Q.total = (f4 ? 16 : 4) * tail;
      if (s == TM_OK) s = fire(pl, kind, f4 ? 2 : 1, Q);
    } else {
      s = fire(pl, kind, ccfg, P);
    }
    if (s != TM_OK) return s;
  }
  return TM_OK;
}

// Fused small-matrix path (bf16): a matrix qualifies when k <= 128 and its
// padded Y, A and B fit in the 160 KB of LDS of one compute unit.
constexpr uint64_t kSmallLdsBig = 160u * 1024u;   // variants of the fused kernel
constexpr uint64_t kSmallLdsLow = 64u * 1024u;    // (two workgroups per compute unit)

bool small_eligible(const Item& it) {
  return it.k <= uint32_t(tmk::kSmallMaxK) && tmk::small_lds_bytes(it.k, it.N) <= kSmallLdsBig;
}

// Every iteration of every matrix in one launch per (kp / 32, LDS variant)
// class and per chunk of kMaxSmallEntries entries / kMaxSmallPtrs pointers;
// consecutive single matrices of one shape share a kPtrTab entry.  No
// workspace: everything between reading X and writing the result stays in LDS.
tm_status plan_small(const Plan& pl, int iters, const float* coeffs, int precond) {
  const std::vector<Item>& items = *pl.items;
  for (int F = 1; F <= tmk::kSmallMaxK / 32; ++F)
    for (int big = 0; big < 2; ++big) {
      std::vector<size_t> idx;
      for (size_t i = 0; i < items.size(); ++i) {
        const Item& it = items[i];
        if (int(tmk::small_kp(it.k) / 32u) == F &&
            int(tmk::small_lds_bytes(it.k, it.N) > kSmallLdsLow) == big)
          idx.push_back(i);
      }
      size_t i = 0;
      while (i < idx.size()) {
        tmk::SmallPhase P;
        std::memset(&P, 0, sizeof(P));
        P.iters = iters;
        P.precond = precond;
        for (int t = 0; t < iters; ++t) {
          P.coef[t][0] = coeffs ? coeffs[3 * t] : kA;
          P.coef[t][1] = coeffs ? coeffs[3 * t + 1] : kB;
          P.coef[t][2] = coeffs ? coeffs[3 * t + 2] : kC;
        }
        uint64_t start = 0;
        int xp = 0;
        while (i < idx.size() && P.nent < tmk::kMaxSmallEntries) {
          const Item& it = items[idx[i]];
          Entry& E = P.e[P.nent];
          E.x = it.x;
          E.k = it.k;
          E.N = it.N;
          E.kp = tmk::small_kp(it.k);
          E.Np = tmk::small_np(it.N);
          E.flags = it.tall ? tmk::kTall : 0u;
          E.tile_start = uint32_t(start);
          E.tiles_per = 1u;
          E.count = it.count;
          ++i;
          // a run of single matrices of this shape: one pointer-table entry
          auto same = [&](size_t j) {
            const Item& v = items[idx[j]];
            return it.count == 1u && v.count == 1u && v.k == it.k && v.N == it.N && v.tall == it.tall;
          };
          if (i < idx.size() && same(i) && xp + 2 <= tmk::kMaxSmallPtrs) {
            E.flags |= tmk::kPtrTab;
            E.xbase = uint32_t(xp);
            P.xp[xp++] = it.x;
            while (i < idx.size() && same(i) && xp < tmk::kMaxSmallPtrs) P.xp[xp++] = items[idx[i++]].x;
            E.count = uint32_t(xp) - E.xbase;
          }
          start += E.count;
          ++P.nent;
          if (start >= (uint64_t(1) << 31))
            return fail(TM_ERR_UNSUPPORTED, "too many matrices in one launch");
        }
        P.total = int32_t(start);
        TimedLaunch tl{int(tmk::kKindSmall), nullptr, nullptr};
        if (g_timing && pl.timed) {
          if (hipEventCreate(&tl.start) != hipSuccess || hipEventCreate(&tl.stop) != hipSuccess)
            return fail(TM_ERR_HIP, "hipEventCreate failed");
          (void)hipEventRecord(tl.start, pl.st);
        }
        const hipError_t e = tmk::launch_small_bf16(F, big, P, pl.st);
        if (tl.start) {
          (void)hipEventRecord(tl.stop, pl.st);
          g_timed.push_back(tl);
        }
        if (e != hipSuccess) return fail(TM_ERR_HIP, std::string("kernel launch: ") + hipGetErrorString(e));
      }
    }
  return TM_OK;
}

// Scale vector s from the first Gram (its flags carry the row partials):
// AOL (Algorithm 2, second line) s_i = 1 / sqrt(row sum of |A0|); Schatten-4
// the uniform ||A0||_F^(-1/2), summed from the squares' row partials.  `part`
// is the column granularity of the row partials.
tm_status gram_scale(const Plan& pl, int precond, int part) {
  if (precond == TM_PRECOND_AOL)
    return launch(pl, tmk::kKindAolVector, 0, 0, 0, 0.f, 0.f, 0.f, 0u, part);
  tm_status s = launch(pl, tmk::kKindFrob, 0, 0, 0, 0.f, 0.f, 0.f, tmk::kFromPart, part);
  if (s == TM_OK)
    s = launch(pl, tmk::kKindAolVector, 0, 0, 0, 0.f, 0.f, 0.f, tmk::kFrob | tmk::kS4, 0);
  return s;
}

// Row-partial flags of the first Gram for a pre-conditioning.
uint32_t first_gram_flags(int precond) {
  if (precond == TM_PRECOND_AOL) return tmk::kRowSum;
  if (precond == TM_PRECOND_SCHATTEN4) return tmk::kRowSum | tmk::kRowSq;
  return 0u;
}

// bf16: zero-padded tiled workspace, matrix-core kernels of tm_fast.hip.
tm_status plan_bf16(const Plan& pl, int iters, const float* coeffs, int precond, int tcfg) {
  const bool frob = precond == TM_PRECOND_FROBENIUS;
  const bool from_gram = precond == TM_PRECOND_AOL || precond == TM_PRECOND_SCHATTEN4;
  const bool scaled = from_gram || frob;
  const uint32_t rflags = first_gram_flags(precond);
  const int gcfg1 = choose_sym_cfg(tmk::kKindGram, tcfg, *pl.items);   // with row partials
  const int gcfg = choose_sym_cfg(tmk::kKindGram, tcfg, *pl.items, true);
  const int pcfg = choose_sym_cfg(tmk::kKindPoly, tcfg, *pl.items, true);
  const int part = tmk::kMinTile;   // the matrix-core Gram emits row partials per 64 columns
  // AOL with at most 16 row partials per row: the rescale pass sums s itself
  // (same order as the AOL-vector kernel), one launch fewer per call
  const bool fuse_s = precond == TM_PRECOND_AOL &&
                      std::all_of(pl.items->begin(), pl.items->end(),
                                  [&](const Item& it) { return it.kp <= uint32_t(16 * part); });
  tm_status s = TM_OK;
  if (iters > 0 || from_gram)
    s = launch(pl, tmk::kKindLoadIn, 0, 0, 0, 0.f, 0.f, 0.f, 0u, 0, kCoverCopied);
  if (s == TM_OK && frob) {  // Algorithm 1, first line: s = 1 / ||X0||_F
    s = launch(pl, tmk::kKindFrob, 0, 0, 0, 0.f, 0.f, 0.f, 0u, 0);
    if (s == TM_OK) s = launch(pl, tmk::kKindAolVector, 0, 0, 0, 0.f, 0.f, 0.f, tmk::kFrob, 0);
  }
  if (s != TM_OK) return s;
  if (iters == 0) {
    if (from_gram) {
      s = launch(pl, tmk::kKindGram, gcfg1, tmk::kSlotFirst, 0, 0.f, 0.f, 0.f, rflags | tmk::kA32, 0);
      if (s == TM_OK) s = gram_scale(pl, precond, part);
      if (s != TM_OK) return s;
    }
    if (scaled) s = launch(pl, tmk::kKindApplyScale, 0, 0, 0, 0.f, 0.f, 0.f, 0u, 0);
    return s;
  }
  int src = tmk::kSlotFirst;
  for (int it = 1; it <= iters && s == TM_OK; ++it) {
    const float a = coeffs ? coeffs[3 * (it - 1)] : kA;
    const float b = coeffs ? coeffs[3 * (it - 1) + 1] : kB;
    const float c = coeffs ? coeffs[3 * (it - 1) + 2] : kC;
    const int dst = it == iters ? tmk::kSlotFinal : (it % 2 == 1 ? tmk::kSlotAlt1 : tmk::kSlotAlt2);
    const bool first = it == 1;
    const uint32_t scale = (first && scaled) ? tmk::kScale : 0u;
    const uint32_t gflags = (first ? rflags : 0u) | (scale ? tmk::kA32 : 0u);
    s = launch(pl, tmk::kKindGram, gflags != 0u ? gcfg1 : gcfg, src, 0, 0.f, 0.f, 0.f, gflags, 0);
    if (s == TM_OK && first && from_gram && !fuse_s) s = gram_scale(pl, precond, part);
    if (s == TM_OK && scale)         // A1 = diag(s) A0 diag(s), one rounding
      s = launch(pl, tmk::kKindScaleA, 0, 0, 0, 0.f, 0.f, 0.f, fuse_s ? tmk::kFuseS : 0u, part);
    // with `scale` the polynomial stores B~ diag(s) and the update reads X0
    if (s == TM_OK) s = launch(pl, tmk::kKindPoly, pcfg, 0, 0, a, b, c, scale, 0);
    if (s == TM_OK) s = launch(pl, tmk::kKindUpdate, tcfg, src, dst, a, b, c, 0u, 0);
    src = dst;
  }
  return s;
}

// fp32: generic kernels of tm_kernels.hip.
tm_status plan_f32(const Plan& pl, int iters, const float* coeffs, int precond) {
  const std::vector<Item>& items = *pl.items;
  tm_status s = TM_OK;
  const bool frob = precond == TM_PRECOND_FROBENIUS;
  const bool from_gram = precond == TM_PRECOND_AOL || precond == TM_PRECOND_SCHATTEN4;
  const bool scaled = from_gram || frob;
  const uint32_t rflags = first_gram_flags(precond);
  bool any_tall = false;
  for (const Item& it : items) any_tall = any_tall || it.tall;
  if (any_tall && (iters > 0 || from_gram)) {
    s = launch(pl, tmk::kKindTransposeIn, 0, 0, 0, 0.f, 0.f, 0.f, 0u, 0, kCoverTall);
    if (s != TM_OK) return s;
  }
  const int gcfg = choose_cfg(tmk::kKindGram, items);
  const int pcfg = choose_cfg(tmk::kKindPoly, items);
  const int ucfg = choose_cfg(tmk::kKindUpdate, items);
  const int part = tmk::cfg_tile(gcfg);   // row partials per Gram tile column block

  if (frob) {  // Algorithm 1, first line: s = 1 / ||X0||_F
    s = launch(pl, tmk::kKindFrob, 0, 0, 0, 0.f, 0.f, 0.f, 0u, 0);
    if (s == TM_OK) s = launch(pl, tmk::kKindAolVector, 0, 0, 0, 0.f, 0.f, 0.f, tmk::kFrob, 0);
    if (s != TM_OK) return s;
  }
  if (iters == 0) {
    if (from_gram) {
      s = launch(pl, tmk::kKindGram, gcfg, tmk::kSlotFirst, 0, 0.f, 0.f, 0.f, rflags | tmk::kA32, 0);
      if (s == TM_OK) s = gram_scale(pl, precond, part);
      if (s != TM_OK) return s;
    }
    if (scaled) s = launch(pl, tmk::kKindApplyScale, 0, 0, 0, 0.f, 0.f, 0.f, 0u, 0);
    return s;
  }

  int src = tmk::kSlotFirst;
  for (int it = 1; it <= iters; ++it) {
    const float a = coeffs ? coeffs[3 * (it - 1)] : kA;
    const float b = coeffs ? coeffs[3 * (it - 1) + 1] : kB;
    const float c = coeffs ? coeffs[3 * (it - 1) + 2] : kC;
    // A single iteration would read and write the caller's buffer: it goes
    // through W1 and a final copy instead.
    const int dst = (it == iters && iters > 1) ? tmk::kSlotFinal
                                               : (it % 2 == 1 ? tmk::kSlotAlt1 : tmk::kSlotAlt2);
    const bool first = it == 1;
    const uint32_t scale = (first && scaled) ? tmk::kScale : 0u;
    const uint32_t gflags = (first ? rflags : 0u) | (scale ? tmk::kA32 : 0u);
    s = launch(pl, tmk::kKindGram, gcfg, src, 0, 0.f, 0.f, 0.f, gflags, 0);
    if (s == TM_OK && first && from_gram) s = gram_scale(pl, precond, part);
    if (s == TM_OK) s = launch(pl, tmk::kKindPoly, pcfg, 0, 0, a, b, c, scale, 0);
    if (s == TM_OK) s = launch(pl, tmk::kKindUpdate, ucfg, src, dst, a, b, c, scale, 0);
    if (s != TM_OK) return s;
    src = dst;
  }
  if (iters == 1) s = launch(pl, tmk::kKindCopyOut, 0, src, 0, 0.f, 0.f, 0.f, 0u, 0);
  return s;
}

// Plan and enqueue one call (g_mu held, device checked).  With ext_ws the
// call runs in that caller-provided device buffer of ext_bytes bytes (the
// allocation-free entry point) instead of the per-stream workspace cache, and
// its launches are never bracketed by the timing hooks' events.
tm_status run_locked(std::vector<Item>& items, int esz, int iters, const float* coeffs,
                     int precond, hipStream_t st, int dev, char* ext_ws = nullptr,
                     uint64_t ext_bytes = 0) {
  tm_status s = TM_OK;
  // bf16 calls made only of small matrices: the fused kernel, one launch
  // (TM_DISABLE_FUSED in the environment keeps them on the tiled kernels)
  if (esz == 2 && iters >= 1 && std::all_of(items.begin(), items.end(), small_eligible) &&
      std::getenv("TM_DISABLE_FUSED") == nullptr) {
    Plan pl;
    pl.items = &items;
    pl.esz = esz;
    pl.st = st;
    pl.ws = nullptr;
    pl.timed = ext_ws == nullptr;
    (void)dev;
    return plan_small(pl, iters, coeffs, precond);
  }
  // A call of more than kMaxEntries items runs every phase as several
  // launches; largest products first, so the last, partly filled launch
  // holds the shortest tiles.  Each matrix's arithmetic does not depend on
  // the launch it lands in.
  if (items.size() > size_t(tmk::kMaxEntries))
    std::stable_sort(items.begin(), items.end(), [](const Item& x, const Item& y) {
      return double(x.k) * x.k * x.N * x.count > double(y.k) * y.k * y.N * y.count;
    });
  int tcfg = 0;
  if (esz == 2) {
    tcfg = choose_tile_cfg(items);
    for (Item& it : items) {
      tmk::tiled_dims(it.k, it.N, uint32_t(tmk::cfg_tile(tcfg)), &it.kp, &it.Np);
      // A wide matrix that needs no padding is read in place by iteration 1;
      // a single iteration would read and write the caller's buffer in the
      // same launch, so it keeps the copy.
      it.direct = !it.tall && it.kp == it.k && it.Np == it.N && iters != 1 &&
                  (reinterpret_cast<uintptr_t>(it.x) & 15u) == 0u;
    }
  } else {
    for (Item& it : items) tmk::generic_dims(it.k, it.N, &it.kp, &it.Np);
  }
  Plan pl;
  pl.items = &items;
  pl.esz = esz;
  pl.st = st;
  pl.tcfg = tcfg;
  uint64_t total = 0;
  for (const Item& it : items) {
    pl.ws_off.push_back(total);
    total += item_ws(it, esz);
  }
  if (total >= (uint64_t(1) << 40))   // entries hold offsets in 256-byte units
    return fail(TM_ERR_UNSUPPORTED, "workspace of more than 1 TB");
  if (ext_ws != nullptr) {
    if (total > ext_bytes)
      return fail(TM_ERR_UNSUPPORTED, "the call needs " + std::to_string(total) +
                                          " bytes of scratch; the static scratch holds " +
                                          std::to_string(ext_bytes));
    pl.ws = ext_ws;
    pl.timed = false;
  } else {
    s = get_workspace(dev, st, size_t(total), &pl.ws);
    if (s != TM_OK) return s;
  }
  return esz == 2 ? plan_bf16(pl, iters, coeffs, precond, tcfg) : plan_f32(pl, iters, coeffs, precond);
}

tm_status run(std::vector<Item>& items, int esz, int iters, const float* coeffs, int precond,
              hipStream_t st) {
  if (items.empty()) return TM_OK;
  std::lock_guard<std::mutex> lock(g_mu);
  int dev = 0;
  tm_status s = check_device(&dev);
  if (s != TM_OK) return s;
  return run_locked(items, esz, iters, coeffs, precond, st, dev);
}

// Enqueue one elementwise optimizer launch per chunk of kMaxOptEntries
// matrices (timed as its own phase when the timing hooks are on).
tm_status launch_opt(int apply, const std::vector<tmk::OptEntry>& ents, const tmk::OptPhase& base,
                     hipStream_t st) {
  for (size_t b0 = 0; b0 < ents.size(); b0 += tmk::kMaxOptEntries) {
    tmk::OptPhase P = base;
    const size_t cnt = std::min(ents.size() - b0, size_t(tmk::kMaxOptEntries));
    uint64_t blocks = 0;
    for (size_t i = 0; i < cnt; ++i) {
      P.e[i] = ents[b0 + i];
      P.e[i].block_start = uint32_t(blocks);
      blocks += (P.e[i].size + tmk::kOptBlock - 1) / tmk::kOptBlock;
    }
    if (blocks >= (uint64_t(1) << 31)) return fail(TM_ERR_UNSUPPORTED, "too many blocks in one launch");
    P.nent = int32_t(cnt);
    P.total = uint32_t(blocks);
    TimedLaunch tl{apply ? int(tmk::kKindOptApply) : int(tmk::kKindOptMomentum), nullptr, nullptr};
    if (g_timing && P.total > 0) {
      if (hipEventCreate(&tl.start) != hipSuccess || hipEventCreate(&tl.stop) != hipSuccess)
        return fail(TM_ERR_HIP, "hipEventCreate failed");
      (void)hipEventRecord(tl.start, st);
    }
    const hipError_t e = tmk::launch_opt(apply, P, st);
    if (tl.start) {
      (void)hipEventRecord(tl.stop, st);
      g_timed.push_back(tl);
    }
    if (e != hipSuccess) return fail(TM_ERR_HIP, std::string("kernel launch: ") + hipGetErrorString(e));
  }
  return TM_OK;
}

tm_status check_common(int iters, const float* coeffs, int precond) {
  if (iters < 0 || iters > TM_MAX_ITERS)
    return fail(TM_ERR_INVALID_ARG, "iters out of range [0, " + std::to_string(TM_MAX_ITERS) + "]");
  if (precond != TM_PRECOND_NONE && precond != TM_PRECOND_FROBENIUS && precond != TM_PRECOND_AOL &&
      precond != TM_PRECOND_SCHATTEN4)
    return fail(TM_ERR_INVALID_ARG, "unknown precond " + std::to_string(precond));
  (void)coeffs;
  return TM_OK;
}

tm_status check_shape(int64_t m, int64_t n) {
  if (m < 1 || n < 1 || m > TM_MAX_DIM || n > TM_MAX_DIM)
    return fail(TM_ERR_INVALID_ARG, "matrix size " + std::to_string(m) + "x" + std::to_string(n) +
                                        " out of range [1, " + std::to_string(TM_MAX_DIM) + "]");
  return TM_OK;
}

Item make_item(void* X, int64_t m, int64_t n, int64_t count) {
  Item it;
  it.x = static_cast<char*>(X);
  it.tall = m > n;
  it.direct = false;
  it.k = uint32_t(std::min(m, n));
  it.N = uint32_t(std::max(m, n));
  it.kp = it.k;
  it.Np = it.N;
  it.count = uint32_t(count);
  return it;
}

tm_status check_batched(void* X, int64_t m, int64_t n, int64_t batch, int iters,
                        const float* coeffs, int precond, int esz) {
  g_last_error.clear();
  tm_status s = check_common(iters, coeffs, precond);
  if (s != TM_OK) return s;
  if (batch < 0) return fail(TM_ERR_INVALID_ARG, "batch < 0");
  s = check_shape(m, n);
  if (s != TM_OK) return s;
  if (batch == 0) return TM_OK;
  if (X == nullptr) return fail(TM_ERR_INVALID_ARG, "X is NULL");
  if (reinterpret_cast<uintptr_t>(X) % uintptr_t(esz) != 0)
    return fail(TM_ERR_UNSUPPORTED, "X is not aligned to its element size");
  if (batch > INT32_MAX) return fail(TM_ERR_INVALID_ARG, "batch too large");
  return TM_OK;
}

tm_status batched(void* X, int64_t m, int64_t n, int64_t batch, int iters, const float* coeffs,
                  int precond, void* stream, int esz) {
  tm_status s = check_batched(X, m, n, batch, iters, coeffs, precond, esz);
  if (s != TM_OK || batch == 0) return s;
  std::vector<Item> items{make_item(X, m, n, batch)};
  return run(items, esz, iters, coeffs, precond, static_cast<hipStream_t>(stream));
}

tm_status grouped(void* const* X, const int64_t* m, const int64_t* n, int64_t count, int iters,
                  const float* coeffs, int precond, void* stream, int esz) {
  g_last_error.clear();
  tm_status s = check_common(iters, coeffs, precond);
  if (s != TM_OK) return s;
  if (count < 0) return fail(TM_ERR_INVALID_ARG, "count < 0");
  if (count == 0) return TM_OK;
  if (X == nullptr || m == nullptr || n == nullptr)
    return fail(TM_ERR_INVALID_ARG, "X, m or n is NULL");
  std::vector<Item> items;
  items.reserve(size_t(count));
  for (int64_t g = 0; g < count; ++g) {
    s = check_shape(m[g], n[g]);
    if (s != TM_OK) return fail(s, "matrix " + std::to_string(g) + ": " + g_last_error);
    if (X[g] == nullptr) return fail(TM_ERR_INVALID_ARG, "X[" + std::to_string(g) + "] is NULL");
    if (reinterpret_cast<uintptr_t>(X[g]) % uintptr_t(esz) != 0)
      return fail(TM_ERR_UNSUPPORTED, "X[" + std::to_string(g) + "] is not element aligned");
    items.push_back(make_item(X[g], m[g], n[g], 1));
  }
  return run(items, esz, iters, coeffs, precond, static_cast<hipStream_t>(stream));
}

}  // namespace

namespace tmk {

// Argument checks of tm_orthogonalize (nothing is enqueued).
tm_status check_batched_bf16(void* X, int64_t m, int64_t n, int64_t batch, int iters,
                             const float* coeffs, int precond) {
  return check_batched(X, m, n, batch, iters, coeffs, precond, 2);
}

// tm_orthogonalize in a caller-provided device buffer `ws` of `ws_bytes`
// (arguments already checked, batch > 0): the same plan and kernels as the
// cached-workspace call, so the results are bitwise equal to it.
tm_status run_batched_bf16_in(void* X, int64_t m, int64_t n, int64_t batch, int iters,
                              const float* coeffs, int precond, void* stream, char* ws,
                              uint64_t ws_bytes) {
  std::vector<Item> items{make_item(X, m, n, batch)};
  std::lock_guard<std::mutex> lock(g_mu);
  int dev = 0;
  tm_status s = check_device(&dev);
  if (s != TM_OK) return s;
  return run_locked(items, 2, iters, coeffs, precond, static_cast<hipStream_t>(stream), dev, ws,
                    ws_bytes);
}

// Record a failure for tm_last_error().
tm_status fail_with(tm_status s, const char* msg) { return fail(s, msg); }

}  // namespace tmk

extern "C" {

tm_status tm_orthogonalize(void* X, int64_t m, int64_t n, int64_t batch, int iters,
                           const float* coeffs, int precond, void* stream) {
  return batched(X, m, n, batch, iters, coeffs, precond, stream, 2);
}

tm_status tm_orthogonalize_f32(float* X, int64_t m, int64_t n, int64_t batch, int iters,
                               const float* coeffs, int precond, void* stream) {
  return batched(X, m, n, batch, iters, coeffs, precond, stream, 4);
}

tm_status tm_orthogonalize_grouped(void* const* X, const int64_t* m, const int64_t* n,
                                   int64_t count, int iters, const float* coeffs, int precond,
                                   void* stream) {
  return grouped(X, m, n, count, iters, coeffs, precond, stream, 2);
}

tm_status tm_orthogonalize_grouped_f32(float* const* X, const int64_t* m, const int64_t* n,
                                       int64_t count, int iters, const float* coeffs,
                                       int precond, void* stream) {
  return grouped(reinterpret_cast<void* const*>(X), m, n, count, iters, coeffs, precond, stream, 4);
}

tm_status tm_muon_step_grouped(float* const* W, const float* const* G, float* const* M,
                               const int64_t* m, const int64_t* n, int64_t count, float lr,
                               float momentum, int nesterov, float weight_decay, int shape_scale,
                               int iters, const float* coeffs, int precond, void* stream) {
  g_last_error.clear();
  tm_status s = check_common(iters, coeffs, precond);
  if (s != TM_OK) return s;
  if (count < 0) return fail(TM_ERR_INVALID_ARG, "count < 0");
  if (count == 0) return TM_OK;
  if (W == nullptr || G == nullptr || M == nullptr || m == nullptr || n == nullptr)
    return fail(TM_ERR_INVALID_ARG, "W, G, M, m or n is NULL");
  for (int64_t g = 0; g < count; ++g) {
    s = check_shape(m[g], n[g]);
    if (s != TM_OK) return fail(s, "matrix " + std::to_string(g) + ": " + g_last_error);
    if (W[g] == nullptr || G[g] == nullptr || M[g] == nullptr)
      return fail(TM_ERR_INVALID_ARG, "matrix " + std::to_string(g) + ": NULL pointer");
    if ((reinterpret_cast<uintptr_t>(W[g]) | reinterpret_cast<uintptr_t>(G[g]) |
         reinterpret_cast<uintptr_t>(M[g])) % 4u != 0)
      return fail(TM_ERR_UNSUPPORTED, "matrix " + std::to_string(g) + ": pointer not 4-byte aligned");
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  std::lock_guard<std::mutex> lock(g_mu);
  int dev = 0;
  s = check_device(&dev);
  if (s != TM_OK) return s;
  uint64_t ubytes = 0;
  for (int64_t g = 0; g < count; ++g) ubytes += tmk::align256(uint64_t(m[g]) * uint64_t(n[g]) * 2u);
  char* ubase = nullptr;
  s = get_workspace(dev, st, size_t(ubytes), &ubase, g_ws_u);
  if (s != TM_OK) return s;
  std::vector<tmk::OptEntry> ents(static_cast<size_t>(count));
  std::vector<Item> items;
  items.reserve(size_t(count));
  uint64_t off = 0;
  for (int64_t g = 0; g < count; ++g) {
    tmk::OptEntry& E = ents[size_t(g)];
    std::memset(&E, 0, sizeof(E));
    E.w = W[g];
    E.g = G[g];
    E.m = M[g];
    E.u = reinterpret_cast<uint16_t*>(ubase + off);
    E.size = uint64_t(m[g]) * uint64_t(n[g]);
    E.vec = ((reinterpret_cast<uintptr_t>(W[g]) | reinterpret_cast<uintptr_t>(G[g]) |
              reinterpret_cast<uintptr_t>(M[g])) & 15u) == 0u;
    E.scale = shape_scale ? std::sqrt(std::max(1.0f, float(m[g]) / float(n[g]))) : 1.0f;
    items.push_back(make_item(E.u, m[g], n[g], 1));
    off += tmk::align256(E.size * 2u);
  }
  tmk::OptPhase base;
  std::memset(&base, 0, sizeof(base));
  base.lr = lr;
  base.mu = momentum;
  base.wd = weight_decay;
  base.nesterov = nesterov ? 1 : 0;
  s = launch_opt(0, ents, base, st);                                          // M, bf16 U
  if (s == TM_OK) s = run_locked(items, 2, iters, coeffs, precond, st, dev);  // U <- O
  if (s == TM_OK) s = launch_opt(1, ents, base, st);                          // W
  return s;
}

const float* tm_schedule_tail(const float* schedule, int rows, int iters) {
  g_last_error.clear();
  if (schedule == nullptr) {
    fail(TM_ERR_INVALID_ARG, "schedule is NULL");
    return nullptr;
  }
  if (rows < 1 || rows > TM_MAX_ITERS || iters < 0 || iters > rows) {
    fail(TM_ERR_INVALID_ARG, "need 1 <= rows <= " + std::to_string(TM_MAX_ITERS) +
                                 " and 0 <= iters <= rows (rows " + std::to_string(rows) +
                                 ", iters " + std::to_string(iters) + ")");
    return nullptr;
  }
  return schedule + 3 * (rows - iters);
}

uint64_t tm_workspace_bytes(const int64_t* m, const int64_t* n, int64_t count, int dtype_bytes) {
  if (m == nullptr || n == nullptr || count < 0 || (dtype_bytes != 2 && dtype_bytes != 4)) return 0;
  std::vector<Item> items;
  for (int64_t g = 0; g < count; ++g) {
    if (m[g] < 1 || n[g] < 1 || m[g] > TM_MAX_DIM || n[g] > TM_MAX_DIM) return 0;
    items.push_back(make_item(nullptr, m[g], n[g], 1));
  }
  if (items.empty()) return 0;
  const int tcfg = dtype_bytes == 2 ? choose_tile_cfg(items) : 0;
  uint64_t total = 0;
  for (Item& it : items) {
    if (dtype_bytes == 2) tmk::tiled_dims(it.k, it.N, uint32_t(tmk::cfg_tile(tcfg)), &it.kp, &it.Np);
    else tmk::generic_dims(it.k, it.N, &it.kp, &it.Np);
    total += item_ws(it, dtype_bytes);
  }
  return total;
}

tm_status tm_release_workspaces(void) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_ws.empty() && g_ws_u.empty() && g_retired.empty()) return TM_OK;
  hipError_t e = hipDeviceSynchronize();
  for (WsCache* c : {&g_ws, &g_ws_u}) {
    for (auto& kv : *c)
      if (kv.second.ptr) (void)hipFree(kv.second.ptr);
    c->clear();
  }
  for (void* p : g_retired) (void)hipFree(p);
  g_retired.clear();
  if (e != hipSuccess) return fail(TM_ERR_HIP, std::string("hipDeviceSynchronize: ") + hipGetErrorString(e));
  return TM_OK;
}

tm_status tm_timing_enable(int enable) {
  std::lock_guard<std::mutex> lock(g_mu);
  g_timing = enable != 0;
  return TM_OK;
}

tm_status tm_timing_read(int phase, double* total_ms, int64_t* launches) {
  if (phase < 0 || phase >= TM_NUM_PHASES || total_ms == nullptr || launches == nullptr)
    return fail(TM_ERR_INVALID_ARG, "bad phase or null output");
  std::lock_guard<std::mutex> lock(g_mu);
  collect_timing();
  *total_ms = g_time_ms[phase];
  *launches = g_time_n[phase];
  return TM_OK;
}

tm_status tm_timing_reset(void) {
  std::lock_guard<std::mutex> lock(g_mu);
  collect_timing();
  for (int i = 0; i < TM_NUM_PHASES; ++i) {
    g_time_ms[i] = 0.0;
    g_time_n[i] = 0;
  }
  return TM_OK;
}

const char* tm_status_string(tm_status s) {
  switch (s) {
    case TM_OK: return "TM_OK";
    case TM_ERR_INVALID_ARG: return "TM_ERR_INVALID_ARG";
    case TM_ERR_UNSUPPORTED: return "TM_ERR_UNSUPPORTED";
    case TM_ERR_NO_MEMORY: return "TM_ERR_NO_MEMORY";
    case TM_ERR_HIP: return "TM_ERR_HIP";
  }
  return "TM_ERR_UNKNOWN";
}

const char* tm_last_error(void) { return g_last_error.c_str(); }

const char* tm_version(void) { return "0.1.0"; }

}  // extern "C"
