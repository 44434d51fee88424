// Internal interface between the host orchestration (lapsum_api.cpp) and the
// HIP kernels.  Every launcher enqueues on `stream` and returns the launch
// status; none synchronises.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace lapsum {

// Largest row solved entirely on chip by one workgroup (keys in LDS).
constexpr int64_t kRowOnChipMax = 32768;
// Tile of the device-wide sort and of the device-wide solve.
constexpr int kTileThreads = 256;
constexpr int kTileItems = 16;
constexpr int64_t kTile = kTileThreads * kTileItems;   // 4096
// Bracketed pass: blocks of the streaming partition and their staging.
constexpr int kPartThreads = 256;
constexpr int kPartMaxBlocks = 4096;   // blocks of the streaming partition
constexpr int kPartStageCap = 960;     // M entries a partition block stages (LDS: 5 blocks per CU)
constexpr int kSelectBins = 2048;      // 11-bit digits of the order-statistic select
constexpr int kSelectGroups = 64;      // coarse groups of kSelectBins / kSelectGroups bins
constexpr int kSampleCntWords = kSelectBins / 2 + kSelectGroups;   // scnt words per sample block

// Threshold record written by the device-wide solve (one per row).
struct SolveRec {
  double b;
  double lap_aL;   // LapSum(a_L) from the scan totals (bracketed only)
  double lap_aR;   // LapSum(a_R)
  int32_t ok;      // bracket certified (always 1 for a full sort)
  int32_t side;    // 0 certified, +1 b >= a_R (LapSum(a_R) > k), -1 b < a_L
};

// Per-block record of the streaming partition (64 bytes; the first 16 are
// what the bucketed solve needs of every block: one aligned load).
struct alignas(16) PartBlock {
  float mmin, mmax;   // smallest / largest member of M (+inf / -inf if none)
  int32_t nM;
  int32_t overflow;   // this block's M did not fit its staging
  int64_t nL, nR;
  double TL, TR;
  int64_t band_dense;   // 1: this block's band lists are incomplete
  int64_t pad;
};
static_assert(sizeof(PartBlock) == 64, "PartBlock layout");

// Totals of the streaming partition (one per attempt).
struct PartTotals {
  int64_t nL, nM, nR;
  double TL, TR;
  float aL, aR;       // the bracket that was partitioned
  float mmin, mmax;   // range of M (+inf / -inf when M is empty)
  int32_t any_block_overflow;
  int32_t dense_blocks;   // partition blocks whose band lists are incomplete
};

// Band of a bracket: the scores whose p depends on where b falls inside a
// certified bracket [a_L, a_R].  With lo = a_L - 105 t (rounded down to
// float32) and hi = a_R + 18 t (rounded up), every score below lo has
// (r - b)/t < -104 and p exactly 0 in float32, and every score at or above
// hi has (r - b)/t > 17 and p exactly 1, for any b in the bracket.  The
// partition stages the band in index order and records, per tile of
// kBandTile scores, where the tile's members sit in the lists; the dense
// writers then fill p (and grad_r) tile by tile without re-reading r, and
// the backward visits only the band.  A row where a quarter or more of the
// blocks could not list their band is instead streamed whole by the emit
// and the backward (the saved header then says mode 1).
constexpr double kBandLowT = 105.0;
constexpr double kBandHighT = 18.0;
constexpr int kBandWaveCapMax = 512;        // band entries a partition wave stages
constexpr int64_t kBandMaxChunk = 65536;    // longer block ranges take the dense passes
constexpr int64_t kBandTile = 1024;         // scores per tile of the dense writers

struct alignas(8) BandEntry {
  int32_t idx;     // index in the row
  uint32_t bits;   // float32 score
};

// Per partition block.
struct BandBlock {
  int32_t cnt[4];   // band members met by each wave (can exceed the capacity)
  int32_t dense;    // 1: the lists of this block are incomplete; passes read it densely
  int32_t pad[3];
};

// Where the members of one tile are: entries [first, first + count) of the
// list array, in index order; count -1 when the tile takes the dense form
// (its block's lists are incomplete).
struct BandTile {
  int32_t first;
  int32_t count;
};

// Saved band of one row (the forward's context for the backward).
struct CtxHeader {
  int32_t mode;     // 0: band lists valid; 1: no lists, every pass is dense
  int32_t nblocks;
  int64_t chunk;
  int32_t cap;      // entries per wave segment
  int32_t pad;
  int64_t n;
  double b;         // the forward's root (mode 0)
};

struct BandCtx {
  CtxHeader* hdr;
  BandBlock* blk;    // [nblocks]
  BandTile* tiles;   // [ceil(n / kBandTile)]
  BandEntry* ent;    // [nblocks][4][cap]
  int nblocks;
  int64_t chunk;
  int cap;
};

// Order statistics of the noised sample.
struct SelectRec {
  float aL, aR;
  uint32_t keyL, keyR;
};

// Optional per-kernel event timing (lapsum_profile_*): a no-op unless on.
void prof_begin(const char* name, hipStream_t s);
void prof_end(hipStream_t s);
struct ProfScope {
  hipStream_t s;
  ProfScope(const char* name, hipStream_t st) : s(st) { prof_begin(name, st); }
  ~ProfScope() { prof_end(s); }
};

// -------------------------------------------------------------- launchers --
hipError_t launch_fill_u32(uint32_t* dst, int64_t count, uint32_t value, hipStream_t s);

// Full-sort forward for rows with n <= kRowOnChipMax (one workgroup per row).
// gated: only rows whose b holds NaN (left by launch_row_bucket_forward) are
// solved; the others exit at once.
hipError_t launch_row_forward(const float* scores, int64_t batch, int64_t n, double k, double t,
                              float* p, double* b, int32_t* perm, bool gated, hipStream_t s);
// The same threshold and p for rows with n <= kRowOnChipMax without sorting
// them (bucketed solve, bucket_solve.hip); a row it cannot finish gets
// b = NaN and no p (the gated launch_row_forward completes it).
hipError_t launch_row_bucket_forward(const float* scores, int64_t batch, int64_t n, double k,
                                     double t, float* p, double* b, hipStream_t s);
// Backward for rows with n <= kRowOnChipMax; grad_k / grad_alpha ([batch]
// float64, each may be null) receive the budget and temperature gradients.
hipError_t launch_row_backward(const float* grad_p, const float* p, int64_t batch, int64_t n,
                               double t, float* grad_r, double* grad_k, double* grad_alpha,
                               hipStream_t s);

// Comparators (comparator_kernels.hip).  Bisection baseline: one thread per
// row, `steps` float32 bisection steps on the plain sum, then p.
hipError_t launch_bisect(const float* r, int64_t batch, int64_t n, double k, double t, int steps,
                         float* p, double* b, hipStream_t s);
// DFTopK on one row: c and the boundary pair from the descending sort
// (keys, source positions), the logistic emit, and the backward (partials:
// dftopk_blocks(n) doubles).
int dftopk_blocks(int64_t n);
hipError_t launch_dftopk_pick(const uint32_t* keys, const int32_t* vals, int64_t k, double* c,
                              int32_t* pair, hipStream_t s);
hipError_t launch_dftopk_emit(const float* r, int64_t n, const double* c, double t, float* p,
                              hipStream_t s);
hipError_t launch_dftopk_backward(const float* g, const float* p, int64_t n, const int32_t* pair,
                                  double t, double* partials, float* grad, hipStream_t s);

// Hard top-k mask from a descending order: mask[row][perm[row][j]] = (j < k).
hipError_t launch_topk_mask(const int32_t* perm, int64_t batch, int64_t n, int64_t k, float* mask,
                            hipStream_t s);

// Laplace-CDF emit p = sigma((r - b)/t) for one row, b read from device.
hipError_t launch_emit(const float* r, int64_t n, const double* b_dev, double t, float* p,
                       hipStream_t s);

// Device-wide backward for one row: partial sums per block, reduced in a
// fixed order to coef[0] = <g, q> and coef[1] = 1/t (0 when sum f == 0),
// then the emit.  The partials are (sum s, sum s g), or with grad_k /
// grad_alpha requested (sum s, sum s g, sum s u, sum s g u) with
// s = min(p, 1 - p), u = (r - b)/t; partials holds 4 doubles per block.
// grad_k / grad_alpha: one float64 each (may be null).  With many partials
// one block combines them into coef (launched by launch_vjp_reduce); with
// few, every emit block combines them itself and coef is not used.  Both
// calls take the same nblocks / nparts and grad_k / grad_alpha.
int vjp_reduce_blocks(int64_t n);
hipError_t launch_vjp_reduce(const float* g, const float* p, int64_t n, double* partials,
                             int nblocks, double t, double* coef, double* grad_k,
                             double* grad_alpha, hipStream_t s);
hipError_t launch_vjp_emit(const float* g, const float* p, int64_t n, const double* coef,
                           const double* partials, int nparts, double t, double* grad_k,
                           double* grad_alpha, float* grad, hipStream_t s);

// Device-wide stable LSD radix sort (descending float order) of one array.
// Source: floats (converted to keys) or keys; values: none, the source
// position, or an int32 array.  len_dev (nullable) overrides len with a
// device-side length <= len.
struct SortBuffers {
  uint32_t* keys[2];
  int32_t* vals[2];
  uint32_t* hist;      // [256][max_tiles]
  uint32_t* totals;    // [256]
  int64_t max_tiles;
};
size_t sort_hist_words(int64_t len);
int64_t sort_max_tiles(int64_t len);
// pass_mask: bit p set when pass p (bits 8p..8p+7) must run; a pass whose
// digit every key shares may be left out (a float source always runs its
// first requested pass).  *keys_out / *vals_out point at the sorted result
// (the source itself when no pass ran).
hipError_t launch_sort(const float* src_f, const uint32_t* src_k, const int32_t* src_v,
                       bool with_vals, int64_t len, const int64_t* len_dev, SortBuffers& sb,
                       unsigned pass_mask, const uint32_t** keys_out, const int32_t** vals_out,
                       hipStream_t s);

// Device-wide threshold solve on a sorted (descending keys) array with the
// bracket tails as carries.  nR/aR/TR: scores ranked before the array; aL/TL:
// after it (T == 0 or +-inf anchors mean none).  n_total: row length.
struct SolveArgs {
  const uint32_t* keys;
  int64_t len;
  const int64_t* len_dev;   // nullable
  double k, t;
  int64_t n_total;
  // tails (bracketed); full sort passes zeros / infinities
  const PartTotals* tails;  // nullable => no tails
  double* tile_buf;         // kSolveTileDoubles per tile
  int64_t max_tiles;
  SolveRec* out;
  double* b_out;            // nullable: also store b here
};
constexpr int kSolveTileDoubles = 8;
hipError_t launch_sorted_solve(const SolveArgs& a, hipStream_t s);

// Bracketed pipeline.
// ykeys: [K]; soffs: [sample_blocks(K) * (kSelectBins + 1)]; scnt:
// [sample_blocks(K) * kSampleCntWords] (per block the bin counts packed two
// to a word, then the counts of the kSelectGroups groups of bins); the
// sample also clears zero[0 .. zero_words) for passes that accumulate later.
int sample_blocks(int64_t K);
// idx: null (systematic sample) or [K] indices of the i.i.d. sample.
// The sample's noise: the caller's table, or (table null) the counter-based
// Laplace(0, t) draws of `seed` (counter_laplace).
struct NoiseSrc {
  const float* table;
  uint64_t seed;
};
hipError_t launch_sample(const float* r, int64_t n, NoiseSrc noise, double t, const int32_t* idx,
                         int64_t K, uint32_t* ykeys, uint32_t* soffs, uint32_t* scnt, uint32_t* zero,
                         int64_t zero_words, hipStream_t s);
// The table counter_laplace gives for draws 0..K-1 of `seed`.
hipError_t launch_noise_table(uint64_t seed, int64_t K, double t, float* out, hipStream_t s);
hipError_t launch_select(const uint32_t* ykeys, int64_t K, const uint32_t* soffs,
                         const uint32_t* scnt, int64_t j, int64_t l, SelectRec* out,
                         hipStream_t s);
int partition_blocks(int64_t n, int64_t* chunk);
int band_wave_cap(int64_t chunk);
// Bytes of one row's context and its layout at `base` (null base: sizes only).
size_t band_ctx_bytes(int64_t n);
BandCtx band_ctx_view(void* base, int64_t n);
// ones: [ceil(n / kBandTile) * kBandTile / 32] bit set where r >= hi (written
// only when a_R is finite; the words past n are never written).  has_r: a_R
// is finite (with use_sel, the selected rank l is at most K); a false has_r
// with a finite a_R would leave R uncounted.
hipError_t launch_partition(const float* r, int64_t n, const SelectRec* sel, int use_sel, float aL,
                            float aR, bool has_r, double t, int nblocks, int64_t chunk,
                            float* stage_v, int32_t* stage_i, PartBlock* blk, const BandCtx& band,
                            uint32_t* ones, hipStream_t s);
// Fixed-order totals of the block records (*tot) and each block's offset
// into M (for launch_gather).
hipError_t launch_partition_totals(const PartBlock* blk, int nblocks, const SelectRec* sel,
                                   int use_sel, float aL, float aR, int64_t* offsets,
                                   PartTotals* tot, hipStream_t s);
// Emit after a certified bracket (skipped when rec->ok == 0): p of every
// score, from the band lists and the ones bits (used when tot->aR is
// finite), and from r for tiles without usable lists; b_out[0] = rec->b; the
// context header is set (with b).
hipError_t launch_band_emit(const float* r, int64_t n, const SolveRec* rec, double t,
                            const BandCtx& band, const uint32_t* ones, const PartTotals* tot,
                            float* p, double* b_out, hipStream_t s);
// Mark a context as dense (rows solved by the full sort).
hipError_t launch_ctx_dense(const BandCtx& band, int64_t n, hipStream_t s);
// Backward from a saved band: partial (sum f, sum f g) per run of blocks,
// then grad_r written densely (zero outside the band).  partials: 4 doubles
// per part, band_vjp_parts(nblocks) parts; gstash: one float per list slot.
// grad_k / grad_alpha (one float64 each, may be null) receive the budget and
// temperature gradients; requesting either adds sum s u and sum s g u to the
// partials.
int band_vjp_parts(int nblocks);
hipError_t launch_band_vjp(const float* g, const float* p, int64_t n, const BandCtx& band,
                           float* gstash, double* partials, double t, float* grad,
                           double* grad_k, double* grad_alpha, hipStream_t s);
hipError_t launch_gather(const float* r, int64_t n, const PartTotals* tot, const PartBlock* blk,
                         const int64_t* offsets, int nblocks, int64_t chunk, const float* stage_v,
                         const int32_t* stage_i, int64_t m_capacity, uint32_t* m_keys,
                         int32_t* m_idx, hipStream_t s);
// |M| <= kRowOnChipMax: sort M on chip, certify and solve in one workgroup.
hipError_t launch_small_m_solve(const uint32_t* m_keys, const int32_t* m_idx, int64_t m_len,
                                bool with_idx, const PartTotals* tot, double k, double t,
                                int64_t n_total, SolveRec* out, int32_t* m_idx_sorted,
                                hipStream_t s);
// Middle set solved by buckets of keys (only the bucket holding the root is
// sorted), straight from the partition's staging: count block c takes the
// staged M of partition blocks [c g, (c+1) g) with g =
// bucket_group_size(nblocks) (at most kBucketGroup), and the
// solve also forms the partition totals (*tot) in a fixed order.  acc:
// bucket accumulators, zero on entry and left zero (keys, offs, parts:
// scratch).  The record reports ok = 0 with side = 2 when the root's bucket
// exceeds kBucketSortCap keys and side = 3 when a block's staging
// overflowed or |M| exceeds m_cap; the caller then gathers M in index order
// and solves it by the full sort.
constexpr int kBucketCount = 2048;
constexpr int kBucketSortCap = 4096;
constexpr int kBucketGroup = 128;   // most partition blocks per count block
// One count block's share of the partition totals, and the range and size
// of all of M (the same in every count block).
struct alignas(16) CountPart {
  double TL, TR;
  int64_t nL, nR, nM;
  int32_t overflow;   // a block of this group overflowed its staging
  uint32_t kmin, kmax;   // keys of max M and min M over every block
  int32_t any_overflow;
  int64_t m_all;
  int32_t ndense;   // blocks of this group whose band lists are incomplete
  int32_t pad;
};
struct BucketAcc {
  uint32_t* n;              // [kBucketCount]
  unsigned long long* u;    // [kBucketCount]
  unsigned long long* d;    // [kBucketCount]
  uint32_t* keys;           // [bucket_keys_words(nblocks)] M per count block in bucket order
  uint32_t* offs;           // [bucket_offs_words(nblocks)] bucket offsets per count block
  CountPart* parts;         // [bucket_groups(nblocks)]
};
constexpr int64_t kBucketAccWords = kBucketCount * 5;   // u32 words of n, u, d
int bucket_group_size(int nblocks);
int bucket_groups(int nblocks);
size_t bucket_keys_words(int nblocks);
size_t bucket_offs_words(int nblocks);
struct PartSource {
  const PartBlock* blk;
  int nblocks;
  const float* stage_v;      // [nblocks * kPartStageCap]
  const SelectRec* sel;      // the bracket: sel (use_sel) or aL, aR
  int use_sel;
  float aL, aR;
};
// The totals of a partition and the record of its solve, next to each other
// so that one copy (or one write to host memory) brings both back.
struct AttemptRec {
  PartTotals tot;
  SolveRec rec;
};
// host: null, or a device-visible pointer to host memory that also receives
// the totals and the record, after which host_seq (same memory) is set to
// seq (a system-scope fence between): the host polls it, no event or copy
// sits on the stream.
hipError_t launch_bucket_solve(const PartSource& ps, int64_t m_cap, BucketAcc acc, PartTotals* tot,
                               double k, double t, int64_t n_total, SolveRec* out,
                               AttemptRec* host, uint32_t* host_seq, uint32_t seq, hipStream_t s);

// Copy sorted M indices to the caller's [m_capacity] row, -1 padded.
hipError_t launch_write_m_idx(const int32_t* sorted_idx, int64_t m_len, int64_t m_capacity,
                              int32_t* out, hipStream_t s);

}  // namespace lapsum
