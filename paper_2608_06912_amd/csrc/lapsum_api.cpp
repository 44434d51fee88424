// Host side of liblapsum.so: argument validation, workspace carving, path
// selection and launch order.  Compiled without floating-point contraction
// so that the bracket ranks of Eq. (8) are evaluated exactly as written.
#include <math.h>
#include <string.h>

#include <atomic>
#include <chrono>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/lapsum.h"
#include "kernels.hpp"

using namespace lapsum;

// ------------------------------------------------------- kernel timing ----
namespace {
struct ProfRec {
  const char* name;
  hipEvent_t a, b;
};
struct ProfAgg {
  std::string name;
  int64_t launches;
  double total_ms;
};
bool g_prof_on = false;
std::vector<ProfRec> g_prof_recs;
std::vector<hipEvent_t> g_prof_pool;
size_t g_prof_pool_used = 0;
std::vector<ProfAgg> g_prof_aggs;

hipEvent_t prof_event() {
  if (g_prof_pool_used == g_prof_pool.size()) {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    g_prof_pool.push_back(e);
  }
  return g_prof_pool[g_prof_pool_used++];
}
}  // namespace

namespace lapsum {
void prof_begin(const char* name, hipStream_t s) {
  if (!g_prof_on) return;
  ProfRec r{name, prof_event(), prof_event()};
  if (r.a && r.b && hipEventRecord(r.a, s) == hipSuccess) g_prof_recs.push_back(r);
}
void prof_end(hipStream_t s) {
  if (!g_prof_on || g_prof_recs.empty()) return;
  // a launch whose end could not be marked is not reported
  if (hipEventRecord(g_prof_recs.back().b, s) != hipSuccess) g_prof_recs.pop_back();
}
}  // namespace lapsum

namespace {

constexpr size_t kAlign = 256;

// Bump allocator over the caller's workspace; a null base only measures.
struct Carve {
  char* base;
  size_t off = 0;
  explicit Carve(void* b) : base(static_cast<char*>(b)) {}
  template <typename T>
  T* take(size_t count) {
    off = (off + kAlign - 1) / kAlign * kAlign;
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
  size_t size() const { return (off + kAlign - 1) / kAlign * kAlign; }
};

int64_t tiles_of(int64_t len) { return (len + kTile - 1) / kTile; }

// ------------------------------------------------------------ device check --
int check_device() {
  static std::mutex mu;
  static int known[64] = {0};   // 0 unknown, 1 gfx950, 2 other
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return LAPSUM_ERR_HIP;
  if (dev < 0 || dev >= 64) return LAPSUM_ERR_DEVICE;
  std::lock_guard<std::mutex> g(mu);
  if (known[dev] == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return LAPSUM_ERR_HIP;
    known[dev] = (strncmp(prop.gcnArchName, "gfx950", 6) == 0) ? 1 : 2;
  }
  return known[dev] == 1 ? LAPSUM_OK : LAPSUM_ERR_DEVICE;
}

bool valid_common(int64_t batch, int64_t n, double k, double alpha) {
  if (batch < 1 || n < 1 || n > 2147483647LL) return false;
  if (!isfinite(k) || !(k > 0.0) || !(k < static_cast<double>(n))) return false;
  if (!isfinite(alpha) || !(alpha < 0.0)) return false;
  return true;
}

int check_ws(void* ws, size_t have, size_t need) {
  if (need == 0) return LAPSUM_OK;
  if (ws == nullptr || have < need) return LAPSUM_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(ws) % kAlign != 0) return LAPSUM_ERR_WORKSPACE;
  return LAPSUM_OK;
}

#define LAPSUM_TRY(expr)                         \
  do {                                           \
    if ((expr) != hipSuccess) return LAPSUM_ERR_HIP; \
  } while (0)

// --------------------------------------------------- full-sort long rows --
struct FullWs {
  SortBuffers sb;
  int64_t solve_tiles;
  double* tile_buf;
  SolveRec* rec;
};

FullWs carve_full(Carve& c, int64_t n, bool with_vals) {
  FullWs w{};
  const int64_t tiles = tiles_of(n) < 1 ? 1 : tiles_of(n);
  w.sb.keys[0] = c.take<uint32_t>(n);
  w.sb.keys[1] = c.take<uint32_t>(n);
  w.sb.vals[0] = with_vals ? c.take<int32_t>(n) : nullptr;
  w.sb.vals[1] = with_vals ? c.take<int32_t>(n) : nullptr;
  w.sb.hist = c.take<uint32_t>(sort_hist_words(n));
  w.sb.totals = c.take<uint32_t>(256);
  w.sb.max_tiles = sort_max_tiles(n);
  w.solve_tiles = tiles;
  w.tile_buf = c.take<double>(static_cast<size_t>(tiles) * kSolveTileDoubles);
  w.rec = c.take<SolveRec>(1);
  return w;
}

// Sort one long row, solve for b (written to b_row), optionally copy the
// permutation.  Does not emit.
int full_row_solve(const float* r, int64_t n, double k, double t, double* b_row, int32_t* perm_row,
                   FullWs& w, hipStream_t s) {
  const uint32_t* keys = nullptr;
  const int32_t* vals = nullptr;
  LAPSUM_TRY(launch_sort(r, nullptr, nullptr, perm_row != nullptr, n, nullptr, w.sb, 0xfu, &keys,
                         &vals, s));
  SolveArgs a{};
  a.keys = keys;
  a.len = n;
  a.len_dev = nullptr;
  a.k = k;
  a.t = t;
  a.n_total = n;
  a.tails = nullptr;
  a.tile_buf = w.tile_buf;
  a.max_tiles = w.solve_tiles;
  a.out = w.rec;
  a.b_out = b_row;
  LAPSUM_TRY(launch_sorted_solve(a, s));
  if (perm_row)
    LAPSUM_TRY(hipMemcpyAsync(perm_row, vals, static_cast<size_t>(n) * sizeof(int32_t),
                              hipMemcpyDeviceToDevice, s));
  return LAPSUM_OK;
}

// --------------------------------------------------------------- bracket --
struct BracketWs {
  uint32_t* ykeys;
  uint32_t* soffs;
  uint32_t* scnt;
  uint32_t* hist;      // the bucket accumulators' words
  BucketAcc acc;
  SelectRec* sel;
  PartBlock* blk;
  int64_t* offsets;
  AttemptRec* att;
  PartTotals* tot;     // &att->tot
  float* stage_v;
  int32_t* stage_i;
  uint32_t* m_keys;
  int32_t* m_idx;
  int32_t* m_idx_sorted;
  SortBuffers msb;     // device-wide sort of M (|M| > on-chip limit)
  int64_t m_solve_tiles;
  double* m_tile_buf;
  SolveRec* rec;       // &att->rec
  FullWs fall;         // full-sort fallback
  uint32_t* ones;      // [ceil(n/kBandTile) kBandTile/32] scores at or above the band (finite a_R)
  void* band;          // one row's band when the caller keeps none
  int nblocks;
  int64_t chunk;
};

BracketWs carve_bracket(Carve& c, int64_t n, int64_t K, int64_t mcap, bool with_idx) {
  BracketWs w{};
  w.nblocks = partition_blocks(n, &w.chunk);
  w.ykeys = c.take<uint32_t>(K);
  // the sample's bin offsets per block, and the bucket accumulators (which
  // the sample clears)
  w.soffs = c.take<uint32_t>(static_cast<size_t>(sample_blocks(K)) * (kSelectBins + 1));
  w.scnt = c.take<uint32_t>(static_cast<size_t>(sample_blocks(K)) * kSampleCntWords);
  w.hist = c.take<uint32_t>(kBucketAccWords);
  w.acc.n = w.hist;
  w.acc.u = reinterpret_cast<unsigned long long*>(w.hist + kBucketCount);
  w.acc.d = reinterpret_cast<unsigned long long*>(w.hist + 3 * kBucketCount);
  w.acc.keys = c.take<uint32_t>(bucket_keys_words(w.nblocks));
  w.acc.offs = c.take<uint32_t>(bucket_offs_words(w.nblocks));
  w.acc.parts = c.take<CountPart>(static_cast<size_t>(bucket_groups(w.nblocks)));
  w.sel = c.take<SelectRec>(1);
  w.blk = c.take<PartBlock>(w.nblocks);
  w.offsets = c.take<int64_t>(w.nblocks);
  w.att = c.take<AttemptRec>(1);
  w.tot = w.att ? &w.att->tot : nullptr;
  w.stage_v = c.take<float>(static_cast<size_t>(w.nblocks) * kPartStageCap);
  w.stage_i = c.take<int32_t>(static_cast<size_t>(w.nblocks) * kPartStageCap);
  w.m_keys = c.take<uint32_t>(mcap);
  w.m_idx = c.take<int32_t>(mcap);
  w.m_idx_sorted = with_idx ? c.take<int32_t>(mcap < kRowOnChipMax ? mcap : kRowOnChipMax) : nullptr;
  if (mcap > kRowOnChipMax) {
    const int64_t mt = tiles_of(mcap);
    w.msb.keys[0] = c.take<uint32_t>(mcap);
    w.msb.keys[1] = c.take<uint32_t>(mcap);
    w.msb.vals[0] = with_idx ? c.take<int32_t>(mcap) : nullptr;
    w.msb.vals[1] = with_idx ? c.take<int32_t>(mcap) : nullptr;
    w.msb.hist = c.take<uint32_t>(sort_hist_words(mcap));
    w.msb.totals = c.take<uint32_t>(256);
    w.msb.max_tiles = sort_max_tiles(mcap);
    w.m_solve_tiles = mt;
    w.m_tile_buf = c.take<double>(static_cast<size_t>(mt) * kSolveTileDoubles);
  }
  w.rec = w.att ? &w.att->rec : nullptr;
  if (n > kRowOnChipMax) w.fall = carve_full(c, n, false);
  w.ones = c.take<uint32_t>(static_cast<size_t>((n + kBandTile - 1) / kBandTile * (kBandTile / 32)));
  w.band = c.take<char>(band_ctx_bytes(n));
  return w;
}

size_t bracketed_ws(int64_t n, int64_t K, int64_t mcap, bool with_idx) {
  Carve c(nullptr);
  carve_bracket(c, n, K, mcap, with_idx);
  return c.size();
}

// Descending uint32 key of a float (the device's order-preserving map).
uint32_t host_desc_key(float f) {
  uint32_t u;
  memcpy(&u, &f, sizeof(u));
  const uint32_t asc = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ~asc;
}

// LSD passes a sort of keys within [key(mmax), key(mmin)] needs: the leading
// bytes both ends share are shared by every key in between.
unsigned sort_pass_mask(float mmin, float mmax) {
  if (!(mmin <= mmax)) return 0xfu;
  const uint32_t lo = host_desc_key(mmax), hi = host_desc_key(mmin);
  unsigned mask = 0xfu;
  for (int p = 3; p >= 0; --p) {
    if (((lo >> (8 * p)) & 255u) != ((hi >> (8 * p)) & 255u)) break;
    mask &= ~(1u << p);
  }
  return mask;
}

// Eq. (8) in IEEE float64, left to right, no contraction.
void bracket_ranks(int64_t n, double k, int64_t K, double z, int64_t* j, int64_t* l) {
  const double q = (static_cast<double>(n) - k) / static_cast<double>(n);
  const double Kq = static_cast<double>(K) * q;
  const double var = Kq * (1.0 - q);
  const double sd = sqrt(var);
  const double zs = z * sd;
  *j = static_cast<int64_t>(floor(Kq - zs));
  *l = static_cast<int64_t>(ceil(Kq + zs));
}

// One-sided doubling, float64 on the float32 endpoints, rounded to float32.
void widen(float* aL, float* aR, int side) {
  const double L = *aL, R = *aR;
  const double w = R - L;
  if (side > 0) {
    *aL = static_cast<float>(R);
    *aR = static_cast<float>(R + 2.0 * w);
  } else {
    *aL = static_cast<float>(L - 2.0 * w);
    *aR = static_cast<float>(L);
  }
}

// Pinned host records the bracketed path reads back (one set per host
// thread, allocated on its first use and kept; one slot per row in flight),
// and the event that tells the host a copy has landed while later work
// proceeds on the stream.
struct HostStage {
  AttemptRec att;
  uint32_t seq;   // set by the bucketed solve after att
  uint32_t pad[3];
};
// Rows of a batch whose first bracket is enqueued before the host reads
// the first row's record (each with its own workspace slice and host slot).
constexpr int kRowsInFlight = 4;
struct ThreadStage {
  HostStage* h = nullptr;
  HostStage* dev = nullptr;   // the same memory as the device addresses it
  hipEvent_t ev = nullptr;
  uint32_t next_seq = 1;
};
thread_local ThreadStage t_stage;

// Mapped, coherent pinned memory: the bucketed solve writes its record there
// directly, so that no copy has to run on the stream before the emit.
int host_stage(HostStage** h, HostStage** dev, hipEvent_t* ev) {
  if (!t_stage.h) {
    void* ptr = nullptr;
    if (hipHostMalloc(&ptr, kRowsInFlight * sizeof(HostStage),
                      hipHostMallocPortable | hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess)
      return LAPSUM_ERR_HIP;
    void* dptr = nullptr;
    if (hipHostGetDevicePointer(&dptr, ptr, 0) != hipSuccess) return LAPSUM_ERR_HIP;
    t_stage.h = static_cast<HostStage*>(ptr);
    t_stage.dev = static_cast<HostStage*>(dptr);
    for (int i = 0; i < kRowsInFlight; ++i) t_stage.h[i].seq = 0u;
  }
  if (!t_stage.ev) {
    if (hipEventCreateWithFlags(&t_stage.ev, hipEventDisableTiming) != hipSuccess)
      return LAPSUM_ERR_HIP;
  }
  *h = t_stage.h;
  *dev = t_stage.dev;
  *ev = t_stage.ev;
  return LAPSUM_OK;
}

// Copy one record to pinned host memory and mark it with the event; the
// caller may enqueue more work before waiting.
template <typename T>
int copy_back(T* host, const T* dev, hipEvent_t ev, hipStream_t s) {
  if (hipMemcpyAsync(host, dev, sizeof(T), hipMemcpyDeviceToHost, s) != hipSuccess) return LAPSUM_ERR_HIP;
  if (hipEventRecord(ev, s) != hipSuccess) return LAPSUM_ERR_HIP;
  return LAPSUM_OK;
}

int wait_back(hipEvent_t ev) {
  return hipEventSynchronize(ev) == hipSuccess ? LAPSUM_OK : LAPSUM_ERR_HIP;
}

// Poll the sequence number a kernel sets in mapped host memory after its
// record.  The stream is queried only once the number has been missing for a
// few milliseconds: a query on a stream whose last command is a kernel makes
// the runtime enqueue a marker behind that kernel, and the marker's cache
// writeback delays the next kernel by several microseconds.  If the stream
// has finished (or failed) without the number appearing, the call fails
// instead of waiting on; so does a wait longer than kSeqWaitLimit (a bracket
// attempt takes well under a millisecond per 1e8 scores, so only work that
// can no longer finish, or a stream held up by other work, reaches it).
constexpr std::chrono::seconds kSeqWaitLimit(30);

int wait_seq(const HostStage* h, uint32_t want, hipStream_t s) {
  const volatile uint32_t* seq = &h->seq;
  using clock = std::chrono::steady_clock;
  const auto start = clock::now();
  bool patient = true;
  for (uint64_t i = 1;; ++i) {
    if (*seq == want) {
      std::atomic_thread_fence(std::memory_order_acquire);
      return LAPSUM_OK;
    }
    if ((i & 255u) != 0u) continue;
    if (patient) {
      if (clock::now() - start < std::chrono::milliseconds(4)) continue;
      patient = false;
    }
    if ((i & 1023u) != 0u) continue;
    const hipError_t q = hipStreamQuery(s);
    if (q == hipErrorNotReady) {
      if (clock::now() - start > kSeqWaitLimit) return LAPSUM_ERR_HIP;
      continue;
    }
    if (q == hipSuccess && *seq == want) {
      std::atomic_thread_fence(std::memory_order_acquire);
      return LAPSUM_OK;
    }
    return LAPSUM_ERR_HIP;
  }
}

// The first bracket of a row without requested M indices: sample, select,
// partition, bucketed solve (its record and then `seq` to host slot
// `slot`), and the emit, which writes p only if the bracket was certified.
// Nothing waits; bracketed_row takes the row from there.
int launch_first_bracket(const float* r, int64_t n, double k, double alpha, int64_t K, double z,
                         NoiseSrc noise, const int32_t* sample_idx, int64_t mcap,
                         float* p_row, double* b_row, void* band_row, BracketWs& w, int slot,
                         uint32_t seq, hipStream_t s) {
  const double t = -alpha;
  HostStage* hs = nullptr;
  HostStage* hs_dev = nullptr;
  hipEvent_t ev = nullptr;
  const int st = host_stage(&hs, &hs_dev, &ev);
  if (st != LAPSUM_OK) return st;
  int64_t j = 0, l = 0;
  bracket_ranks(n, k, K, z, &j, &l);
  const BandCtx band = band_ctx_view(band_row ? band_row : w.band, n);
  LAPSUM_TRY(launch_sample(r, n, noise, t, sample_idx, K, w.ykeys, w.soffs, w.scnt, w.hist,
                           kBucketAccWords, s));
  LAPSUM_TRY(launch_select(w.ykeys, K, w.soffs, w.scnt, j, l, w.sel, s));
  LAPSUM_TRY(launch_partition(r, n, w.sel, 1, 0.0f, 0.0f, l <= K, t, w.nblocks, w.chunk,
                              w.stage_v, w.stage_i, w.blk, band, w.ones, s));
  const PartSource ps{w.blk, w.nblocks, w.stage_v, w.sel, 1, 0.0f, 0.0f};
  LAPSUM_TRY(launch_bucket_solve(ps, mcap, w.acc, w.tot, k, t, n, w.rec, &hs_dev[slot].att,
                                 &hs_dev[slot].seq, seq, s));
  LAPSUM_TRY(launch_band_emit(r, n, w.rec, t, band, w.ones, w.tot, p_row, b_row, s));
  return LAPSUM_OK;
}

// A first bracket already enqueued by launch_first_bracket.
struct FirstBracket {
  int slot;
  uint32_t seq;
};

int bracketed_row(const float* r, int64_t n, double k, double alpha, int64_t K, double z,
                  NoiseSrc noise, const int32_t* sample_idx, int64_t mcap, int64_t out_cap, uint32_t flags, float* p_row,
                  double* b_row, lapsum_bracket_info* info, int32_t* midx_row, void* band_row,
                  BracketWs& w, hipStream_t s, const FirstBracket* pre = nullptr) {
  const double t = -alpha;
  lapsum_bracket_info rec_info;
  memset(&rec_info, 0, sizeof(rec_info));
  int64_t j = 0, l = 0;
  bracket_ranks(n, k, K, z, &j, &l);
  rec_info.j = j;
  rec_info.l = l;
  bool solved = false;
  bool wrote_midx = false;
  const BandCtx band = band_ctx_view(band_row ? band_row : w.band, n);
  HostStage* hs = nullptr;
  HostStage* hs_dev = nullptr;
  hipEvent_t ev = nullptr;
  int st = host_stage(&hs, &hs_dev, &ev);
  if (st != LAPSUM_OK) return st;
  if (pre) hs += pre->slot;   // this row's record lands in its own slot

  if (!(flags & LAPSUM_FLAG_FULL_SORT)) {
    if (!pre) {
      LAPSUM_TRY(launch_sample(r, n, noise, t, sample_idx, K, w.ykeys, w.soffs, w.scnt, w.hist,
                               kBucketAccWords, s));
      LAPSUM_TRY(launch_select(w.ykeys, K, w.soffs, w.scnt, j, l, w.sel, s));
    }
    float aL = 0.0f, aR = 0.0f;
    const bool want_idx = midx_row != nullptr;
    for (int attempt = 1; attempt <= 3 && !solved; ++attempt) {
      const int use_sel = attempt == 1 ? 1 : 0;
      const bool prelaunched = pre && attempt == 1;   // partition, solve and emit enqueued
      if (!prelaunched)
        LAPSUM_TRY(launch_partition(r, n, w.sel, use_sel, aL, aR,
                                    use_sel ? l <= K : aR < INFINITY, t, w.nblocks, w.chunk,
                                    w.stage_v, w.stage_i, w.blk, band, w.ones, s));
      // M in index order, one contiguous array: needed for the sorted
      // indices and for the full sort of M; the buckets read the staging
      auto gather_in_order = [&]() -> int {
        LAPSUM_TRY(launch_partition_totals(w.blk, w.nblocks, w.sel, use_sel, aL, aR, w.offsets,
                                           w.tot, s));
        LAPSUM_TRY(launch_gather(r, n, w.tot, w.blk, w.offsets, w.nblocks, w.chunk, w.stage_v,
                                 w.stage_i, mcap, w.m_keys, w.m_idx, s));
        return LAPSUM_OK;
      };
      const int32_t* sorted_idx = nullptr;
      PartTotals tot;
      // M by sorting all of it (needed for the sorted indices, or when the
      // buckets cannot take it); |M| known on the host
      auto solve_sorted = [&]() -> int {
        if (tot.nM <= kRowOnChipMax) {
          LAPSUM_TRY(launch_small_m_solve(w.m_keys, w.m_idx, tot.nM, want_idx, w.tot, k, t, n,
                                          w.rec, w.m_idx_sorted, s));
          sorted_idx = w.m_idx_sorted;
        } else {
          const uint32_t* mk = nullptr;
          const int32_t* mv = nullptr;
          LAPSUM_TRY(launch_sort(nullptr, w.m_keys, w.m_idx, want_idx, tot.nM, nullptr, w.msb,
                                 sort_pass_mask(tot.mmin, tot.mmax), &mk, &mv, s));
          SolveArgs a{};
          a.keys = mk;
          a.len = tot.nM;
          a.len_dev = nullptr;
          a.k = k;
          a.t = t;
          a.n_total = n;
          a.tails = w.tot;
          a.tile_buf = w.m_tile_buf;
          a.max_tiles = w.m_solve_tiles;
          a.out = w.rec;
          a.b_out = nullptr;
          LAPSUM_TRY(launch_sorted_solve(a, s));
          sorted_idx = want_idx ? mv : nullptr;
        }
        return LAPSUM_OK;
      };
      // the records come back to the host while the emit runs; the emit (and
      // its write of b) happens only if this bracket was certified
      auto emit_and_read = [&]() -> int {
        int e = copy_back(&hs->att, w.att, ev, s);
        if (e != LAPSUM_OK) return e;
        LAPSUM_TRY(launch_band_emit(r, n, w.rec, t, band, w.ones, w.tot, p_row, b_row, s));
        return wait_back(ev);
      };
      bool have_rec = false;
      if (!want_idx) {
        // buckets straight from the staging, with no wait for the totals
        // the solve writes its record to host memory as well; the emit (of
        // a certified bracket only) runs while the host waits for it
        uint32_t seq = 0;
        if (prelaunched) {
          seq = pre->seq;
        } else {
          const int slot = pre ? pre->slot : 0;
          const PartSource ps{w.blk, w.nblocks, w.stage_v, w.sel, use_sel, aL, aR};
          seq = t_stage.next_seq++;
          LAPSUM_TRY(launch_bucket_solve(ps, mcap, w.acc, w.tot, k, t, n, w.rec,
                                         &hs_dev[slot].att, &hs_dev[slot].seq, seq, s));
          LAPSUM_TRY(launch_band_emit(r, n, w.rec, t, band, w.ones, w.tot, p_row, b_row, s));
        }
        st = wait_seq(hs, seq, s);
        if (st != LAPSUM_OK) return st;
        tot = hs->att.tot;
        have_rec = true;
      } else {
        st = gather_in_order();
        if (st == LAPSUM_OK) st = copy_back(&hs->att, w.att, ev, s);
        if (st == LAPSUM_OK) st = wait_back(ev);
        if (st != LAPSUM_OK) return st;
        tot = hs->att.tot;
      }
      aL = tot.aL;
      aR = tot.aR;
      rec_info.attempts = attempt;
      rec_info.a_L = tot.aL;
      rec_info.a_R = tot.aR;
      rec_info.n_L = tot.nL;
      rec_info.n_M = tot.nM;
      rec_info.n_R = tot.nR;
      rec_info.T_L = tot.TL;
      rec_info.T_R = tot.TR;
      if (tot.nM > mcap) {
        // no room for M: the certificate is never evaluated
        rec_info.m_overflow = 1;
        rec_info.lap_aL = NAN;
        rec_info.lap_aR = NAN;
        break;
      }
      if (!have_rec || (!hs->att.rec.ok && hs->att.rec.side >= 2)) {
        st = have_rec ? gather_in_order() : LAPSUM_OK;
        if (st == LAPSUM_OK) st = solve_sorted();
        if (st == LAPSUM_OK) st = emit_and_read();
        if (st != LAPSUM_OK) return st;
      }
      const SolveRec rec = hs->att.rec;
      rec_info.lap_aL = rec.lap_aL;
      rec_info.lap_aR = rec.lap_aR;
      if (rec.ok) {
        if (want_idx) {
          LAPSUM_TRY(launch_write_m_idx(sorted_idx, tot.nM, out_cap, midx_row, s));
          wrote_midx = true;
        }
        solved = true;
        break;
      }
      if (attempt < 3) widen(&aL, &aR, rec.side);
    }
  }
  if (!solved) {
    rec_info.fell_back = 1;
    if (n <= kRowOnChipMax) {
      // the on-chip kernel also emits p
      LAPSUM_TRY(launch_row_forward(r, 1, n, k, t, p_row, b_row, nullptr, false, s));
    } else {
      st = full_row_solve(r, n, k, t, b_row, nullptr, w.fall, s);
      if (st != LAPSUM_OK) return st;
      LAPSUM_TRY(launch_emit(r, n, b_row, t, p_row, s));
    }
    LAPSUM_TRY(launch_ctx_dense(band, n, s));
  }
  if (midx_row && !wrote_midx) LAPSUM_TRY(launch_write_m_idx(nullptr, 0, out_cap, midx_row, s));
  if (info) *info = rec_info;
  return LAPSUM_OK;
}


struct DftopkWs {
  SortBuffers sb;
  double* partials;
};

DftopkWs carve_dftopk(Carve& c, int64_t n) {
  DftopkWs w{};
  w.sb.keys[0] = c.take<uint32_t>(n);
  w.sb.keys[1] = c.take<uint32_t>(n);
  w.sb.vals[0] = c.take<int32_t>(n);
  w.sb.vals[1] = c.take<int32_t>(n);
  w.sb.hist = c.take<uint32_t>(sort_hist_words(n));
  w.sb.totals = c.take<uint32_t>(256);
  w.sb.max_tiles = sort_max_tiles(n);
  w.partials = c.take<double>(static_cast<size_t>(dftopk_blocks(n)));
  return w;
}

bool dftopk_args(int64_t batch, int64_t n, int64_t k, double alpha) {
  return batch >= 1 && n >= 2 && n <= 2147483647LL && k >= 1 && k < n && isfinite(alpha) &&
         alpha < 0.0;
}

}  // namespace

extern "C" {

int lapsum_profile_start(void) {
  g_prof_recs.clear();
  g_prof_aggs.clear();
  g_prof_pool_used = 0;
  g_prof_on = true;
  return LAPSUM_OK;
}

int lapsum_profile_stop(void) {
  g_prof_on = false;
  std::map<std::string, size_t> where;
  for (const ProfRec& r : g_prof_recs) {
    if (hipEventSynchronize(r.b) != hipSuccess) return -LAPSUM_ERR_HIP;
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return -LAPSUM_ERR_HIP;
    auto it = where.find(r.name);
    if (it == where.end()) {
      where[r.name] = g_prof_aggs.size();
      g_prof_aggs.push_back(ProfAgg{r.name, 1, static_cast<double>(ms)});
    } else {
      g_prof_aggs[it->second].launches += 1;
      g_prof_aggs[it->second].total_ms += ms;
    }
  }
  g_prof_recs.clear();
  g_prof_pool_used = 0;
  return static_cast<int>(g_prof_aggs.size());
}

int lapsum_profile_entry(int i, char* name, size_t name_len, int64_t* launches, double* total_ms) {
  if (i < 0 || static_cast<size_t>(i) >= g_prof_aggs.size() || !name || name_len == 0)
    return LAPSUM_ERR_INVALID_ARG;
  const ProfAgg& a = g_prof_aggs[static_cast<size_t>(i)];
  strncpy(name, a.name.c_str(), name_len - 1);
  name[name_len - 1] = '\0';
  if (launches) *launches = a.launches;
  if (total_ms) *total_ms = a.total_ms;
  return LAPSUM_OK;
}

const char* lapsum_status_string(int status) {
  switch (status) {
    case LAPSUM_OK: return "ok";
    case LAPSUM_ERR_INVALID_ARG: return "invalid argument";
    case LAPSUM_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    case LAPSUM_ERR_HIP: return "HIP runtime or launch error";
    case LAPSUM_ERR_DEVICE: return "current device is not gfx950";
    default: return "unknown status";
  }
}

// One workgroup per row sorts rows of up to kRowOnChipMax scores on chip,
// all rows of a batch at once.  A single row longer than kRowSingleMax
// leaves most of the chip idle that way and goes through the device-wide
// sort instead (measured on MI355X: n = 32768 alone takes 0.122 ms on one
// workgroup against 0.072 ms device-wide; at 16384 the two are even).
constexpr int64_t kRowSingleMax = 16384;

bool forward_on_chip(int64_t batch, int64_t n) {
  return n <= kRowOnChipMax && !(batch == 1 && n > kRowSingleMax);
}

size_t lapsum_forward_workspace_size(int64_t batch, int64_t n, int with_perm) {
  if (n < 1) return 0;
  if (forward_on_chip(batch, n)) return 0;
  Carve c(nullptr);
  carve_full(c, n, with_perm != 0);
  return c.size();
}

int lapsum_forward(const float* scores, int64_t batch, int64_t n, double k, double alpha, float* p,
                   double* b, int32_t* perm_out, void* workspace, size_t workspace_bytes,
                   hipStream_t stream) {
  if (!scores || !p || !b || !valid_common(batch, n, k, alpha)) return LAPSUM_ERR_INVALID_ARG;
  const int wst = check_ws(workspace, workspace_bytes,
                           lapsum_forward_workspace_size(batch, n, perm_out != nullptr));
  if (wst != LAPSUM_OK) return wst;
  const int dst = check_device();
  if (dst != LAPSUM_OK) return dst;
  const double t = -alpha;
  if (forward_on_chip(batch, n)) {
    if (perm_out) {
      LAPSUM_TRY(launch_row_forward(scores, batch, n, k, t, p, b, perm_out, false, stream));
    } else {
      // no order wanted: the bucketed solve, then the full sort only for
      // rows it left unsolved.  It leaves a row only when the root's bucket
      // holds more than kBucketSortCap scores, which a shorter row cannot
      // have, so short rows need no second launch.
      LAPSUM_TRY(launch_row_bucket_forward(scores, batch, n, k, t, p, b, stream));
      if (n > kBucketSortCap)
        LAPSUM_TRY(launch_row_forward(scores, batch, n, k, t, p, b, nullptr, true, stream));
    }
    return LAPSUM_OK;
  }
  Carve c(workspace);
  FullWs w = carve_full(c, n, perm_out != nullptr);
  for (int64_t row = 0; row < batch; ++row) {
    const float* r = scores + row * n;
    int st = full_row_solve(r, n, k, t, b + row, perm_out ? perm_out + row * n : nullptr, w, stream);
    if (st != LAPSUM_OK) return st;
    LAPSUM_TRY(launch_emit(r, n, b + row, t, p + row * n, stream));
  }
  return LAPSUM_OK;
}

size_t lapsum_backward_workspace_size(int64_t batch, int64_t n) {
  (void)batch;
  if (n <= kRowOnChipMax) return 0;
  Carve c(nullptr);
  c.take<double>(4 * static_cast<size_t>(vjp_reduce_blocks(n)));
  c.take<double>(2);
  return c.size();
}

int lapsum_backward(const float* grad_p, const float* p, const double* b, int64_t batch, int64_t n,
                    double alpha, float* grad_r, double* grad_k, double* grad_alpha,
                    void* workspace, size_t workspace_bytes, hipStream_t stream) {
  (void)b;
  if (!grad_p || !p || !grad_r) return LAPSUM_ERR_INVALID_ARG;
  if (batch < 1 || n < 1 || n > 2147483647LL || !isfinite(alpha) || !(alpha < 0.0))
    return LAPSUM_ERR_INVALID_ARG;
  const int wst = check_ws(workspace, workspace_bytes, lapsum_backward_workspace_size(batch, n));
  if (wst != LAPSUM_OK) return wst;
  const int dst = check_device();
  if (dst != LAPSUM_OK) return dst;
  const double t = -alpha;
  if (n <= kRowOnChipMax) {
    LAPSUM_TRY(launch_row_backward(grad_p, p, batch, n, t, grad_r, grad_k, grad_alpha, stream));
    return LAPSUM_OK;
  }
  Carve c(workspace);
  const int nb = vjp_reduce_blocks(n);
  double* partials = c.take<double>(4 * static_cast<size_t>(nb));
  double* coef = c.take<double>(2);
  for (int64_t row = 0; row < batch; ++row) {
    const int64_t o = row * n;
    LAPSUM_TRY(launch_vjp_reduce(grad_p + o, p + o, n, partials, nb, t, coef,
                                 grad_k ? grad_k + row : nullptr,
                                 grad_alpha ? grad_alpha + row : nullptr, stream));
    LAPSUM_TRY(launch_vjp_emit(grad_p + o, p + o, n, coef, partials, nb, t,
                               grad_k ? grad_k + row : nullptr,
                               grad_alpha ? grad_alpha + row : nullptr, grad_r + o, stream));
  }
  return LAPSUM_OK;
}

int lapsum_topk_mask(const int32_t* perm, int64_t batch, int64_t n, int64_t k, float* mask,
                     hipStream_t stream) {
  if (!perm || !mask || batch < 1 || n < 1 || n > 2147483647LL || k < 0 || k > n)
    return LAPSUM_ERR_INVALID_ARG;
  const int dst = check_device();
  if (dst != LAPSUM_OK) return dst;
  LAPSUM_TRY(launch_topk_mask(perm, batch, n, k, mask, stream));
  return LAPSUM_OK;
}

int lapsum_bisect_forward(const float* scores, int64_t batch, int64_t n, double k, double alpha,
                          int32_t steps, float* p, double* b, hipStream_t stream) {
  if (!scores || !p || !b || !valid_common(batch, n, k, alpha) || steps < 0 || steps > 200)
    return LAPSUM_ERR_INVALID_ARG;
  const int dst = check_device();
  if (dst != LAPSUM_OK) return dst;
  LAPSUM_TRY(launch_bisect(scores, batch, n, k, -alpha, steps, p, b, stream));
  return LAPSUM_OK;
}


size_t lapsum_dftopk_workspace_size(int64_t batch, int64_t n) {
  (void)batch;
  if (n < 2 || n > 2147483647LL) return 0;
  Carve c(nullptr);
  carve_dftopk(c, n);
  return c.size();
}

int lapsum_dftopk_forward(const float* scores, int64_t batch, int64_t n, int64_t k, double alpha,
                          float* p, double* c_out, int32_t* pair, void* workspace,
                          size_t workspace_bytes, hipStream_t stream) {
  if (!scores || !p || !c_out || !pair || !dftopk_args(batch, n, k, alpha))
    return LAPSUM_ERR_INVALID_ARG;
  const int wst = check_ws(workspace, workspace_bytes, lapsum_dftopk_workspace_size(batch, n));
  if (wst != LAPSUM_OK) return wst;
  const int dst = check_device();
  if (dst != LAPSUM_OK) return dst;
  Carve c(workspace);
  DftopkWs w = carve_dftopk(c, n);
  for (int64_t row = 0; row < batch; ++row) {
    const float* r = scores + row * n;
    const uint32_t* keys = nullptr;
    const int32_t* vals = nullptr;
    LAPSUM_TRY(launch_sort(r, nullptr, nullptr, true, n, nullptr, w.sb, 0xfu, &keys, &vals,
                           stream));
    LAPSUM_TRY(launch_dftopk_pick(keys, vals, k, c_out + row, pair + 2 * row, stream));
    LAPSUM_TRY(launch_dftopk_emit(r, n, c_out + row, -alpha, p + row * n, stream));
  }
  return LAPSUM_OK;
}

int lapsum_dftopk_backward(const float* grad_p, const float* p, const int32_t* pair, int64_t batch,
                           int64_t n, double alpha, float* grad_r, void* workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  if (!grad_p || !p || !pair || !grad_r || !dftopk_args(batch, n, 1, alpha))
    return LAPSUM_ERR_INVALID_ARG;
  const int wst = check_ws(workspace, workspace_bytes, lapsum_dftopk_workspace_size(batch, n));
  if (wst != LAPSUM_OK) return wst;
  const int dst = check_device();
  if (dst != LAPSUM_OK) return dst;
  Carve c(workspace);
  DftopkWs w = carve_dftopk(c, n);
  for (int64_t row = 0; row < batch; ++row) {
    const int64_t o = row * n;
    LAPSUM_TRY(launch_dftopk_backward(grad_p + o, p + o, n, pair + 2 * row, -alpha, w.partials,
                                      grad_r + o, stream));
  }
  return LAPSUM_OK;
}

// Workspace slices of a bracketed call: one per row in flight (rows of a
// batch without requested M indices), each a whole row's workspace.
int64_t bracket_slices(int64_t batch, bool with_idx) {
  return with_idx ? 1 : (batch < kRowsInFlight ? (batch < 1 ? 1 : batch) : kRowsInFlight);
}

size_t lapsum_forward_bracketed_workspace_size(int64_t batch, int64_t n, int64_t K,
                                               int64_t m_capacity, int with_m_idx) {
  if (n < 1 || K < 1 || m_capacity < 1) return 0;
  const size_t one = bracketed_ws(n, K, m_capacity < n ? m_capacity : n, with_m_idx != 0);
  return static_cast<size_t>(bracket_slices(batch, with_m_idx != 0)) * one;
}

size_t lapsum_band_size(int64_t batch, int64_t n) {
  if (batch < 1 || n < 1 || n > 2147483647LL) return 0;
  return static_cast<size_t>(batch) * band_ctx_bytes(n);
}

int lapsum_forward_bracketed(const float* scores, int64_t batch, int64_t n, double k, double alpha,
                             int64_t K, double z, const float* noise_table, uint64_t seed,
                             const int32_t* sample_idx, int64_t m_capacity,
                             uint32_t flags, float* p, double* b, lapsum_bracket_info* info,
                             int32_t* m_idx_out, void* band, size_t band_bytes, void* workspace,
                             size_t workspace_bytes, hipStream_t stream) {
  if (!scores || !p || !b || !valid_common(batch, n, k, alpha)) return LAPSUM_ERR_INVALID_ARG;
  const NoiseSrc noise{noise_table, seed};
  if (K < 2 || K > n || !isfinite(z) || !(z > 0.0) || m_capacity < 1 || (flags & ~LAPSUM_FLAG_FULL_SORT))
    return LAPSUM_ERR_INVALID_ARG;
  if (band && (band_bytes < lapsum_band_size(batch, n) || reinterpret_cast<uintptr_t>(band) % kAlign))
    return LAPSUM_ERR_INVALID_ARG;
  // |M| <= n always, so capacity beyond n is never used internally; the
  // caller's m_idx_out rows keep their m_capacity stride.
  const int64_t mcap = m_capacity < n ? m_capacity : n;
  const bool with_idx = m_idx_out != nullptr;
  const int wst = check_ws(workspace, workspace_bytes,
                           lapsum_forward_bracketed_workspace_size(batch, n, K, m_capacity, with_idx));
  if (wst != LAPSUM_OK) return wst;
  const int dst = check_device();
  if (dst != LAPSUM_OK) return dst;
  const size_t band_row_bytes = band_ctx_bytes(n);
  auto band_of = [&](int64_t row) -> void* {
    return band ? static_cast<char*>(band) + row * band_row_bytes : nullptr;
  };
  Carve c(workspace);
  if (with_idx || (flags & LAPSUM_FLAG_FULL_SORT) || batch == 1) {
    BracketWs w = carve_bracket(c, n, K, mcap, with_idx);
    for (int64_t row = 0; row < batch; ++row) {
      int st = bracketed_row(scores + row * n, n, k, alpha, K, z, noise, sample_idx, mcap,
                             m_capacity, flags, p + row * n, b + row, info ? info + row : nullptr,
                             m_idx_out ? m_idx_out + row * m_capacity : nullptr, band_of(row), w,
                             stream);
      if (st != LAPSUM_OK) return st;
    }
    return LAPSUM_OK;
  }
  // rows in flight: the first brackets of up to kRowsInFlight rows are
  // enqueued before the host reads the first row's record, so the device
  // runs the next rows while the host finishes the earlier ones
  const int64_t P = bracket_slices(batch, false);
  BracketWs ws[kRowsInFlight];
  for (int64_t q = 0; q < P; ++q) ws[q] = carve_bracket(c, n, K, mcap, false);
  FirstBracket pre[kRowsInFlight];
  auto launch = [&](int64_t row) -> int {
    const int q = static_cast<int>(row % P);
    pre[q].slot = q;
    pre[q].seq = t_stage.next_seq++;
    return launch_first_bracket(scores + row * n, n, k, alpha, K, z, noise, sample_idx, mcap,
                                p + row * n, b + row, band_of(row), ws[q], q, pre[q].seq, stream);
  };
  for (int64_t row = 0; row < P; ++row) {
    const int st = launch(row);
    if (st != LAPSUM_OK) return st;
  }
  for (int64_t row = 0; row < batch; ++row) {
    const int q = static_cast<int>(row % P);
    int st = bracketed_row(scores + row * n, n, k, alpha, K, z, noise, sample_idx, mcap,
                           m_capacity, flags, p + row * n, b + row, info ? info + row : nullptr,
                           nullptr, band_of(row), ws[q], stream, &pre[q]);
    if (st == LAPSUM_OK && row + P < batch) st = launch(row + P);
    if (st != LAPSUM_OK) return st;
  }
  return LAPSUM_OK;
}

int lapsum_bracket_noise(uint64_t seed, int64_t K, double alpha, float* out, hipStream_t stream) {
  if (!out || K < 1 || K > 2147483647LL || !isfinite(alpha) || !(alpha < 0.0))
    return LAPSUM_ERR_INVALID_ARG;
  const int dst = check_device();
  if (dst != LAPSUM_OK) return dst;
  LAPSUM_TRY(launch_noise_table(seed, K, -alpha, out, stream));
  return LAPSUM_OK;
}

size_t lapsum_backward_band_workspace_size(int64_t batch, int64_t n) {
  (void)batch;
  if (n < 1 || n > 2147483647LL) return 0;
  const BandCtx v = band_ctx_view(nullptr, n);
  Carve c(nullptr);
  c.take<double>(4 * static_cast<size_t>(band_vjp_parts(v.nblocks)));
  c.take<float>(static_cast<size_t>(v.nblocks) * 4 * v.cap);
  return c.size();
}

int lapsum_backward_band(const float* grad_p, const float* p, const void* band, size_t band_bytes,
                         int64_t batch, int64_t n, double alpha, float* grad_r, double* grad_k,
                         double* grad_alpha, void* workspace, size_t workspace_bytes,
                         hipStream_t stream) {
  if (!grad_p || !p || !band || !grad_r) return LAPSUM_ERR_INVALID_ARG;
  if (batch < 1 || n < 1 || n > 2147483647LL || !isfinite(alpha) || !(alpha < 0.0))
    return LAPSUM_ERR_INVALID_ARG;
  if (band_bytes < lapsum_band_size(batch, n) || reinterpret_cast<uintptr_t>(band) % kAlign)
    return LAPSUM_ERR_INVALID_ARG;
  const int wst = check_ws(workspace, workspace_bytes, lapsum_backward_band_workspace_size(batch, n));
  if (wst != LAPSUM_OK) return wst;
  const int dst = check_device();
  if (dst != LAPSUM_OK) return dst;
  const double t = -alpha;
  const BandCtx v0 = band_ctx_view(nullptr, n);
  Carve c(workspace);
  double* partials = c.take<double>(4 * static_cast<size_t>(band_vjp_parts(v0.nblocks)));
  float* gstash = c.take<float>(static_cast<size_t>(v0.nblocks) * 4 * v0.cap);
  const size_t band_row_bytes = band_ctx_bytes(n);
  for (int64_t row = 0; row < batch; ++row) {
    const int64_t o = row * n;
    // the kernels only read the band
    void* band_row = const_cast<char*>(static_cast<const char*>(band)) + row * band_row_bytes;
    const BandCtx v = band_ctx_view(band_row, n);
    LAPSUM_TRY(launch_band_vjp(grad_p + o, p + o, n, v, gstash, partials, t, grad_r + o,
                               grad_k ? grad_k + row : nullptr,
                               grad_alpha ? grad_alpha + row : nullptr, stream));
  }
  return LAPSUM_OK;
}

}  // extern "C"
