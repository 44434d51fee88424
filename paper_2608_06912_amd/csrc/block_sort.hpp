// Stable LSD radix sort of uint32 keys (optionally with int32 values) held by
// one workgroup in registers, 8-bit digits, scattered through LDS.
//
// Arrangement ("wave-striped"): item i of lane `lane` in wave `w` sits at
// position w*(64*ITEMS) + i*64 + lane.  That position order is the order the
// sort keeps among equal keys, so loading element `pos` of a row into that
// slot makes the sort stable by original index.
//
// Digit ranking per pass: the lanes of a wave holding the same digit are
// found with eight ballots (one per digit bit), giving each lane the number
// of earlier same-digit lanes; a per-wave LDS counter per digit carries the
// count across the ITEMS rounds.  An exclusive scan over the counters in
// digit-major, wave-minor order then gives every (wave, digit) its first
// output position, which keeps the order position-stable.
#pragma once

#include "common.hpp"

namespace lapsum {

__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

// Lanes of this wave whose 8-bit digit equals mine (all 64 lanes active).
// A lane differs from me in bit b exactly where the ballot of bit b differs
// from my bit broadcast to all 64 positions (m = 0 or ~0), so the peers are
// the complement of the OR over the eight bits of (ballot ^ m).  Each bit
// costs one bit-field extract, one compare for the ballot and one
// three-input bit operation per 32-bit half, acc | (ballot ^ m) (truth table
// 0xf6 over the inputs acc, ballot, m), taking the ballot straight from
// scalar registers: 34 vector instructions per match instead of 71 for the
// per-lane select of ballot or its complement.
__device__ __forceinline__ uint64_t match_digit8(uint32_t d) {
  uint32_t lo = 0u, hi = 0u;
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const uint32_t m = static_cast<uint32_t>(__builtin_amdgcn_sbfe(static_cast<int>(d), b, 1));
    const uint64_t bal = __builtin_amdgcn_uicmp(m, 0u, 33);   // 33: integer "not equal"
    lo = __builtin_amdgcn_bitop3_b32(lo, static_cast<uint32_t>(bal), m, 0xf6);
    hi = __builtin_amdgcn_bitop3_b32(hi, static_cast<uint32_t>(bal >> 32), m, 0xf6);
  }
  return (static_cast<uint64_t>(~hi) << 32) | ~lo;
}

// Per-(digit, wave) counters, digit-major.  Each digit's row is padded to an
// odd stride so that the 64 lanes of a wave, which touch the counters of 64
// (mostly different) digits of their own wave at once, spread over all LDS
// banks; with a power-of-two stride they would share very few banks.
template <int WAVES>
__device__ __forceinline__ int cnt_at(uint32_t d, int w) {
  return static_cast<int>(d) * (WAVES + 1) + w;
}
template <int WAVES>
constexpr int cnt_words() { return 256 * (WAVES + 1); }

// In-place exclusive scan, in (digit, wave) order, of the 256 * WAVES
// counters laid out by cnt_at (4 per thread, BLOCK = 64 * WAVES threads).
template <int BLOCK>
__device__ void block_excl_scan_u32x4(uint32_t* a, uint32_t* wave_tot) {
  constexpr int WAVES = BLOCK / kWave;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  int at[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int j = 4 * tid + q;
    at[q] = cnt_at<WAVES>(static_cast<uint32_t>(j / WAVES), j % WAVES);
  }
  uint32_t v0 = a[at[0]], v1 = a[at[1]], v2 = a[at[2]], v3 = a[at[3]];
  uint32_t sum = v0 + v1 + v2 + v3;
  uint32_t incl = sum;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    uint32_t o = __shfl_up(incl, d, kWave);
    if (lane >= d) incl += o;
  }
  if (lane == kWave - 1) wave_tot[wid] = incl;
  __syncthreads();
  uint32_t wbase = 0;
#pragma unroll
  for (int w = 0; w < WAVES; ++w)
    if (w < wid) wbase += wave_tot[w];
  uint32_t ex = wbase + incl - sum;
  a[at[0]] = ex;
  a[at[1]] = ex + v0;
  a[at[2]] = ex + v0 + v1;
  a[at[3]] = ex + v0 + v1 + v2;
  __syncthreads();
}

// The scatter buffer skips one word after every 32 so that the blocked read
// of the last pass (lane stride ITEMS words) does not fall into one bank.
__device__ __forceinline__ int buf_at(int p) { return p + (p >> 5); }
template <int BLOCK, int ITEMS>
constexpr int sort_buf_words() { return BLOCK * ITEMS + (BLOCK * ITEMS) / 32; }

template <int BLOCK>
struct SortSmem {
  uint32_t cnt[cnt_words<BLOCK / kWave>()];
  uint32_t wave_tot[BLOCK / kWave];
};

// One LSD pass on bits [shift, shift+8).  On return the keys (and values)
// are back in registers: wave-striped, or blocked (thread tid holds positions
// tid*ITEMS .. tid*ITEMS+ITEMS-1) when `blocked_out`.  `buf` holds
// sort_buf_words<BLOCK, ITEMS>() u32.
template <int BLOCK, int ITEMS, bool PAIRS>
__device__ void block_sort_pass(uint32_t (&key)[ITEMS], int32_t (&val)[ITEMS], int shift,
                                uint32_t* buf, SortSmem<BLOCK>& sm, bool blocked_out) {
  constexpr int WAVES = BLOCK / kWave;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid / kWave;
  for (int e = tid; e < cnt_words<WAVES>(); e += BLOCK) sm.cnt[e] = 0u;
  __syncthreads();

  uint32_t pos[ITEMS];
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    const uint32_t d = (key[i] >> shift) & 255u;
    const uint64_t peers = match_digit8(d);
    const uint32_t below = lanes_below(peers);
    uint32_t* slot = &sm.cnt[cnt_at<WAVES>(d, wid)];
    const uint32_t c = *slot;
    pos[i] = c + below;
    if (below == 0u) *slot = c + static_cast<uint32_t>(__popcll(peers));
  }
  __syncthreads();
  block_excl_scan_u32x4<BLOCK>(sm.cnt, sm.wave_tot);
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) pos[i] += sm.cnt[cnt_at<WAVES>((key[i] >> shift) & 255u, wid)];

#pragma unroll
  for (int i = 0; i < ITEMS; ++i) buf[buf_at(static_cast<int>(pos[i]))] = key[i];
  __syncthreads();
#pragma unroll
  for (int i = 0; i < ITEMS; ++i)
    key[i] = buf[buf_at(blocked_out ? tid * ITEMS + i : wid * (kWave * ITEMS) + i * kWave + lane)];
  __syncthreads();
  if constexpr (PAIRS) {
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) buf[buf_at(static_cast<int>(pos[i]))] = static_cast<uint32_t>(val[i]);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < ITEMS; ++i)
      val[i] = static_cast<int32_t>(
          buf[buf_at(blocked_out ? tid * ITEMS + i : wid * (kWave * ITEMS) + i * kWave + lane)]);
    __syncthreads();
  }
}

// Full 32-bit sort; the result is left in blocked arrangement.
template <int BLOCK, int ITEMS, bool PAIRS>
__device__ void block_sort_u32(uint32_t (&key)[ITEMS], int32_t (&val)[ITEMS], uint32_t* buf,
                               SortSmem<BLOCK>& sm) {
  block_sort_pass<BLOCK, ITEMS, PAIRS>(key, val, 0, buf, sm, false);
  block_sort_pass<BLOCK, ITEMS, PAIRS>(key, val, 8, buf, sm, false);
  block_sort_pass<BLOCK, ITEMS, PAIRS>(key, val, 16, buf, sm, false);
  block_sort_pass<BLOCK, ITEMS, PAIRS>(key, val, 24, buf, sm, true);
}

}  // namespace lapsum
