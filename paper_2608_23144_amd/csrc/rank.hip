// Gain-ranked record selection and serialization (Eq. (4), Sec. 3.3, Eq. (5)).
//
// With a fixed record size, ordering by rho_t = gain_t / L_rec is ordering by
// gain.  The positive fp64 gains are mapped to their IEEE bit patterns, which
// order like the values.  For a segment of tiles:
//  0. the eligible tiles are counted and K = min(cap, eligible) is formed on
//     the device (the host never waits for it);
//  1. radix select (12-bit digits, most significant first) finds the K-th
//     largest key k* and how many records equal to k* are taken;
//  2. a stable compaction keeps every key > k* and the first such equal keys
//     in tile order (so equal gains keep the lower tile index);
//  3. the K survivors are sorted by (decreasing key, increasing tile): chunks
//     of 256 by a bitonic network in LDS, then multiway merge passes that
//     place each item by searches in the other runs of its group;
//  4. records are bit-packed at fixed offsets h + (first slot of the segment
//     + i) * L_rec.
// Cross-block results only pass between launches.  Each select pass finishes
// the previous pass itself: every block repeats the pick of the bin holding
// the K-th key from the previous histogram (4096 bins, a block scan), so a
// pass is one launch; histograms rotate over three buffers and the pick
// state over two, so no launch overwrites what another block of the same
// launch still reads.  A segment is a chain of launches with no host round
// trip and one read of the totals ends the call.
#include "awsrc_internal.h"

namespace awsrc {

constexpr int kThreads = 256;
constexpr int kRounds = 16;
constexpr int kItems = kThreads * kRounds;  // items per block in the compaction
constexpr int kChunk = 256;                 // items per LDS-sorted chunk
constexpr int kChunkThreads = 128;
constexpr int kLogChunk = 8;
constexpr int kFan = 16;                    // runs per multiway merge
constexpr int kLogFan = 4;
constexpr int kSelBits = 12;                // radix-select digit width
constexpr int kSelBins = 1 << kSelBits;

// Words of RankWs::state.
enum : int {
  kPrefix = 0, kMask = 1, kRem = 2, kDone = 3,  // radix select result of the current segment
  kSegK = 4, kSegOff = 5,                       // records of the segment, its first record slot
  kElig = 6, kArrive = 7,                       // per-launch accumulators, reset after use
  kTotK = 8, kTotElig = 9, kNoSpace = 10,       // totals over the segments of one call
  kSel = 16,                                    // [2][4] pick state of alternate passes
  kHist = 32                                    // [3][kSelBins] histograms of rotating passes
};
static_assert(kHist + 3 * kSelBins == kStateWords, "rank state size");

// Positive doubles order like their bit patterns; the top (sign) bit is set on
// eligible keys so that every eligible key exceeds every ineligible (zero) key.
__device__ __forceinline__ uint64_t gain_key(double g) {
  return g > 0.0 ? ((uint64_t)__double_as_longlong(g) | (1ull << 63)) : 0ull;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & 63;
  return lane ? (~0ull >> (64 - lane)) : 0ull;
}

// Exclusive block scan of a 0/1 flag over kThreads threads; returns the
// exclusive prefix for this thread and the block total in *total.
__device__ __forceinline__ uint32_t block_scan_flag(bool f, uint32_t* sh_w, uint32_t* total) {
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const uint64_t bal = __ballot(f);
  const uint32_t in_wave = __popcll(bal & lanemask_lt());
  if (lane == 0) sh_w[w] = __popcll(bal);
  __syncthreads();
  uint32_t before = 0, tot = 0;
#pragma unroll
  for (int k = 0; k < kThreads / 64; ++k) {
    const uint32_t c = sh_w[k];
    before += (k < w) ? c : 0u;
    tot += c;
  }
  __syncthreads();
  *total = tot;
  return before + in_wave;
}

__global__ void k_rank_init(uint64_t* state) {
  for (int i = threadIdx.x; i < kStateWords; i += blockDim.x) state[i] = 0;
}

// ---------------------------------------------------------------- radix select
// Each pass histograms the next digit of the keys that match the prefix so
// far; the next launch picks the bin holding the remaining-th largest key.
// When that whole bin is taken the search stops early: every key in it is
// selected, so the lower digits no longer matter.

// First pass of a segment, fused with the eligibility count: the top digit
// (eligible flag and exponent) of every key, into histogram 0.
__global__ __launch_bounds__(kThreads) void k_count_hist(const double* __restrict__ gain, int64_t n,
                                                         uint64_t* state) {
  __shared__ uint32_t h[kSelBins];
  __shared__ uint32_t sw[kThreads / 64];
  for (int b = threadIdx.x; b < kSelBins; b += kThreads) h[b] = 0;
  __syncthreads();
  uint32_t c = 0;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  for (; i + 7 * stride < n; i += 8 * stride) {
    double gv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) gv[u] = gain[i + u * stride];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint64_t k = gain_key(gv[u]);
      c += k != 0;
      atomicAdd(&h[k >> (64 - kSelBits)], 1u);
    }
  }
  for (; i < n; i += stride) {
    const uint64_t k = gain_key(gain[i]);
    c += k != 0;
    atomicAdd(&h[k >> (64 - kSelBits)], 1u);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) c += __shfl_xor(c, off, 64);
  if ((threadIdx.x & 63) == 0) sw[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = 0;
    for (int k = 0; k < kThreads / 64; ++k) t += sw[k];
    if (t) atomicAdd((unsigned long long*)&state[kElig], (unsigned long long)t);
  }
  for (int b = threadIdx.x; b < kSelBins; b += kThreads)
    if (h[b]) atomicAdd((unsigned long long*)&state[kHist + b], (unsigned long long)h[b]);
}

struct SelState {
  uint64_t prefix, mask, rem, done;
};

// One block of kThreads: the bin of histogram `hist` (digit at `shift`,
// `width` bits) holding the rem-th largest key; thread t owns bpt consecutive
// bins counted from the top.  Every thread returns the same state.
__device__ SelState pick_bin(const uint64_t* hist, SelState in, int shift, int width) {
  __shared__ uint64_t s_wave[kThreads / 64];
  __shared__ uint64_t found[3];
  constexpr int kMaxBpt = kSelBins / kThreads;
  const int nbins = 1 << width;
  const int bpt = nbins >= kThreads ? nbins / kThreads : 1;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  // this thread's bins, counted from the top, kept in registers for the search
  uint64_t v[kMaxBpt];
  uint64_t local = 0;
#pragma unroll
  for (int i = 0; i < kMaxBpt; ++i) {
    const int r = t * bpt + i;
    v[i] = (i < bpt && r < nbins) ? hist[nbins - 1 - r] : 0ull;
    local += v[i];
  }
  if (t < 3) found[t] = 0;
  // inclusive scan: within the wavefront by shuffles, then across the four
  uint64_t x = local;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_wave[wv] = x;
  __syncthreads();
  uint64_t before = 0;
#pragma unroll
  for (int w = 0; w < kThreads / 64; ++w) before += w < wv ? s_wave[w] : 0ull;
  const uint64_t incl = before + x;
  const uint64_t excl = incl - local;
  if (excl < in.rem && in.rem <= incl) {
    uint64_t cum = excl;
    bool hit = false;
#pragma unroll
    for (int i = 0; i < kMaxBpt; ++i) {
      const uint64_t c = v[i];
      if (!hit && i < bpt && cum + c >= in.rem) {
        found[0] = (uint64_t)(nbins - 1 - (t * bpt + i));
        found[1] = in.rem - cum;
        found[2] = (c == in.rem - cum) ? 1ull : 0ull;
        hit = true;
      }
      cum += c;
    }
  }
  __syncthreads();
  SelState out;
  out.prefix = in.prefix | (found[0] << shift);
  out.mask = in.mask | (((1ull << width) - 1ull) << shift);
  out.rem = found[1];
  out.done = found[2];
  __syncthreads();
  return out;
}

// Pass `pass` (1..5) of a segment: pick from the previous pass's histogram
// (digit at prev_shift), then histogram the next digit (at shift) of the keys
// under the new prefix.  Pass 1 forms K = min(cap, eligible) itself.
__global__ __launch_bounds__(kThreads) void k_select_pass(const double* __restrict__ gain, int64_t n,
                                                          uint64_t* state, int64_t cap, int pass, int prev_shift,
                                                          int prev_width, int shift, int width) {
  __shared__ uint32_t h[kSelBins];
  SelState cur;
  if (pass == 1) {
    const uint64_t ne = state[kElig];
    const uint64_t K = ne < (uint64_t)cap ? ne : (uint64_t)cap;
    cur = SelState{0ull, 0ull, K, K == 0 ? 1ull : 0ull};
    if (blockIdx.x == 0 && threadIdx.x == 0) state[kSegK] = K;
  } else {
    const uint64_t* sp = state + kSel + 4 * ((pass - 1) & 1);
    cur = SelState{sp[0], sp[1], sp[2], sp[3]};
  }
  // the histogram two passes back has been read by the previous launch
  uint64_t* hclr = state + kHist + kSelBins * ((pass + 1) % 3);
  for (int b = blockIdx.x * kThreads + threadIdx.x; b < kSelBins; b += gridDim.x * kThreads) hclr[b] = 0;
  SelState nw = cur;
  if (!cur.done) nw = pick_bin(state + kHist + kSelBins * ((pass - 1) % 3), cur, prev_shift, prev_width);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    uint64_t* so = state + kSel + 4 * (pass & 1);
    so[0] = nw.prefix; so[1] = nw.mask; so[2] = nw.rem; so[3] = nw.done;
  }
  if (nw.done) return;  // uniform
  for (int b = threadIdx.x; b < kSelBins; b += kThreads) h[b] = 0;
  __syncthreads();
  const uint64_t dm = (1ull << width) - 1ull;
  // eight independent loads per thread in flight (the grid is small: each
  // block ends with up to 4096 global atomics)
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  for (; i + 7 * stride < n; i += 8 * stride) {
    double gv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) gv[u] = gain[i + u * stride];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint64_t k = gain_key(gv[u]);
      if ((k & nw.mask) == nw.prefix) atomicAdd(&h[(k >> shift) & dm], 1u);
    }
  }
  for (; i < n; i += stride) {
    const uint64_t k = gain_key(gain[i]);
    if ((k & nw.mask) == nw.prefix) atomicAdd(&h[(k >> shift) & dm], 1u);
  }
  __syncthreads();
  uint64_t* hout = state + kHist + kSelBins * (pass % 3);
  for (int b = threadIdx.x; b < (1 << width); b += kThreads)
    if (h[b]) atomicAdd((unsigned long long*)&hout[b], (unsigned long long)h[b]);
}

// The select result after the last pass (pass 6's pick), as every block of the
// first compaction launch computes it.
__device__ SelState final_select(const uint64_t* state) {
  const uint64_t* sp = state + kSel + 4 * (5 & 1);
  SelState cur = SelState{sp[0], sp[1], sp[2], sp[3]};
  if (!cur.done) cur = pick_bin(state + kHist + kSelBins * (5 % 3), cur, 0, 4);
  return cur;
}

// ---------------------------------------------------------------- compaction
// Every block finishes the select itself (the last pick); block 0 records the
// result, the segment's first record slot and the running totals.
__global__ __launch_bounds__(kThreads) void k_compact_count(const double* __restrict__ gain, int64_t n,
                                                            uint64_t* state, uint64_t* blk_gt, uint64_t* blk_eq) {
  const uint64_t K = state[kSegK];
  const SelState fin = final_select(state);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    state[kPrefix] = fin.prefix;
    state[kMask] = fin.mask;
    state[kRem] = fin.rem;
    state[kDone] = fin.done;
    state[kSegOff] = state[kTotK];
    state[kTotK] += K;
    state[kTotElig] += state[kElig];
    state[kElig] = 0;
  }
  if (K == 0) return;  // uniform
  const uint64_t prefix = fin.prefix, mask = fin.mask;
  uint32_t gt = 0, eq = 0;
  const int64_t base = (int64_t)blockIdx.x * kItems;
  for (int r = 0; r < kRounds; ++r) {
    const int64_t i = base + r * kThreads + threadIdx.x;
    if (i < n) {
      const uint64_t k = gain_key(gain[i]) & mask;
      gt += k > prefix;
      eq += k == prefix;
    }
  }
  __shared__ uint32_t s_gt[kThreads / 64], s_eq[kThreads / 64];
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    gt += __shfl_xor(gt, off, 64);
    eq += __shfl_xor(eq, off, 64);
  }
  if ((threadIdx.x & 63) == 0) { s_gt[threadIdx.x >> 6] = gt; s_eq[threadIdx.x >> 6] = eq; }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t a = 0, b = 0;
    for (int k = 0; k < kThreads / 64; ++k) { a += s_gt[k]; b += s_eq[k]; }
    blk_gt[blockIdx.x] = a;
    blk_eq[blockIdx.x] = b;
  }
}

// Inclusive scan over the 1024 threads of a block: shuffles within each
// wavefront, then the 16 wavefront totals; *total gets the block sum.
__device__ __forceinline__ uint64_t scan1024(uint64_t v, uint64_t* s_wave, uint64_t* total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  uint64_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_wave[wv] = x;
  __syncthreads();
  uint64_t before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < 16; ++w) {
    const uint64_t t = s_wave[w];
    before += w < wv ? t : 0ull;
    tot += t;
  }
  __syncthreads();
  *total = tot;
  return before + x;
}

// Single block: eq offsets (exclusive scan of blk_eq) and selected offsets.
// On exit blk_gt[b] = first output slot of block b, blk_eq[b] = number of
// equal keys in earlier blocks.
__global__ __launch_bounds__(1024) void k_compact_scan(uint64_t* blk_gt, uint64_t* blk_eq, int64_t nblk,
                                                       uint64_t* state) {
  // every histogram has been read: leave them cleared for the next segment
  for (int b = threadIdx.x; b < 3 * kSelBins; b += 1024) state[kHist + b] = 0;
  if (state[kSegK] == 0) return;
  __shared__ uint64_t s_wave[16];
  const uint64_t rem = state[kRem];
  uint64_t carry_eq = 0, carry_sel = 0;
  for (int64_t c0 = 0; c0 < nblk; c0 += 1024) {
    const int64_t i = c0 + threadIdx.x;
    const uint64_t gt = i < nblk ? blk_gt[i] : 0, eq = i < nblk ? blk_eq[i] : 0;
    uint64_t eq_tot, sel_tot;
    const uint64_t eq_excl = carry_eq + scan1024(eq, s_wave, &eq_tot) - eq;
    uint64_t take_eq = 0;
    if (rem > eq_excl) take_eq = (rem - eq_excl) < eq ? (rem - eq_excl) : eq;
    const uint64_t sel = gt + take_eq;
    const uint64_t sel_excl = carry_sel + scan1024(sel, s_wave, &sel_tot) - sel;
    if (i < nblk) { blk_gt[i] = sel_excl; blk_eq[i] = eq_excl; }
    carry_eq += eq_tot;
    carry_sel += sel_tot;
  }
}

// gain: the segment's gains (from tile t0); seed, scale: every tile's
__global__ __launch_bounds__(kThreads) void k_compact_write(const double* __restrict__ gain,
                                                            const uint16_t* __restrict__ seed,
                                                            const uint16_t* __restrict__ scale, int64_t t0, int64_t n,
                                                            const uint64_t* __restrict__ state,
                                                            const uint64_t* __restrict__ sel_off,
                                                            const uint64_t* __restrict__ eq_off,
                                                            SortItem* __restrict__ items_out) {
  if (state[kSegK] == 0) return;  // uniform
  __shared__ uint32_t sh_w[kThreads / 64];
  const uint64_t prefix = state[kPrefix], mask = state[kMask];
  const uint64_t rem = state[kRem];
  uint64_t eq_run = eq_off[blockIdx.x];
  uint64_t sel_run = sel_off[blockIdx.x];
  const int64_t base = (int64_t)blockIdx.x * kItems;
  for (int r = 0; r < kRounds; ++r) {
    const int64_t i = base + r * kThreads + threadIdx.x;
    uint64_t k = 0;
    if (i < n) k = gain_key(gain[i]);
    const bool gt = (i < n) && (k & mask) > prefix;
    const bool eq = (i < n) && (k & mask) == prefix;
    uint32_t eq_tot, sel_tot;
    const uint32_t eq_rank = block_scan_flag(eq, sh_w, &eq_tot);
    const bool take = gt || (eq && (eq_run + eq_rank) < rem);
    const uint32_t pos = block_scan_flag(take, sh_w, &sel_tot);
    if (take) {
      SortItem it;
      it.key = ~k;  // ascending ~key = descending gain
      it.tile = (uint32_t)(t0 + i);
      it.aux = (uint32_t)seed[t0 + i] | ((uint32_t)scale[t0 + i] << 16);
      items_out[sel_run + pos] = it;
    }
    eq_run += eq_tot;
    sel_run += sel_tot;
  }
}

// ---------------------------------------------------------------- packing
struct PackArgs {
  const uint16_t* seed;
  const int8_t* code;
  const uint16_t* scale;
  int P, b, idx_bits, seed_bits, scale_bits, L;
  uint64_t h, cap;
  uint8_t* out;
};

__device__ __forceinline__ void put_bits(uint64_t (&w)[3], int& pos, uint64_t v, int nbits) {
  if (nbits <= 0) return;
  const int o = pos & 63, k = pos >> 6;
  w[k] |= v << o;
  if (o + nbits > 64) w[k + 1] |= v >> (64 - o);
  pos += nbits;
}

// Record i of the segment (tile t) goes to byte h + (first slot + i) * L of
// the stream; a stream buffer too small for the running total raises the
// no-space flag instead.
// Record i of the stream from tile t; aux = the tile's seed | scale << 16.
// A record at a 4-byte aligned place whose size is a multiple of 4 goes out
// as whole words.
__device__ void pack_record(const PackArgs& pa, uint64_t* state, int64_t i, uint32_t t, uint32_t aux) {
  const uint64_t K = state[kSegK], off = state[kSegOff];
  if (pa.h + (off + K) * (uint64_t)pa.L > pa.cap) {
    if (i == 0) state[kNoSpace] = 1;
    return;
  }
  uint64_t w[3] = {0, 0, 0};
  int pos = 0;
  put_bits(w, pos, (uint64_t)t, pa.idx_bits);
  put_bits(w, pos, (uint64_t)(aux & 0xFFFFu), pa.seed_bits);
  const uint64_t cm = (1ull << pa.b) - 1ull;
  for (int p = 0; p < pa.P; ++p) put_bits(w, pos, (uint64_t)(int64_t)pa.code[(int64_t)t * pa.P + p] & cm, pa.b);
  put_bits(w, pos, (uint64_t)(aux >> 16) & ((1ull << pa.scale_bits) - 1ull), pa.scale_bits);
  uint8_t* o = pa.out + pa.h + (off + (uint64_t)i) * (uint64_t)pa.L;
  if (((reinterpret_cast<uintptr_t>(o) | (uintptr_t)pa.L) & 3) == 0) {
    uint32_t* o32 = reinterpret_cast<uint32_t*>(o);
    for (int k = 0; k < pa.L / 4; ++k) o32[k] = (uint32_t)(w[k >> 1] >> (32 * (k & 1)));
  } else {
    for (int k = 0; k < pa.L; ++k) o[k] = (uint8_t)(w[k >> 3] >> (8 * (k & 7)));
  }
}

// the same, with the seed and scale read from the encoder outputs
__device__ __forceinline__ void pack_record(const PackArgs& pa, uint64_t* state, int64_t i, uint32_t t) {
  pack_record(pa, state, i, t, (uint32_t)pa.seed[t] | ((uint32_t)pa.scale[t] << 16));
}

// ---------------------------------------------------------------- sort of the survivors
// Items are (key, tile) pairs; tiles are distinct, so the lexicographic order
// on the pair is a total order and equal gains come out in increasing tile
// order without any stability argument.
__device__ __forceinline__ bool kv_less(const SortItem& a, const SortItem& b) {
  return (a.key < b.key) | ((a.key == b.key) & (a.tile < b.tile));  // no short-circuit branches
}

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// In-place bitonic sort of each chunk of kChunk items in LDS; the tail chunk
// is padded with sentinels that sort last and are not written back.  Pair q of
// a stage with distance j compares elements i = (q with a zero inserted at bit
// log2 j) and i + j; thread t takes pairs t + r kChunkThreads (one pair per
// thread with kChunk = 2 kChunkThreads), so for j <= 64 every wavefront works
// inside its own 128-element windows and a wavefront-level barrier suffices
// between stages.
// With `pack` set (the final pass) the sorted items are packed as records.
__global__ __launch_bounds__(kChunkThreads) void k_sort_chunks(SortItem* __restrict__ items, uint64_t* state,
                                                               int pack, PackArgs pa) {
  __shared__ uint64_t sk[kChunk];
  __shared__ uint32_t st[kChunk];
  const int64_t n = (int64_t)state[kSegK];
  const int64_t base = (int64_t)blockIdx.x * kChunk;
  if (base >= n) return;  // uniform per block
#pragma unroll
  for (int r = 0; r < kChunk / kChunkThreads; ++r) {
    const int j = r * kChunkThreads + threadIdx.x;
    const int64_t i = base + j;
    uint64_t key = ~0ull;
    uint32_t tile = 0xFFFFFFFFu;
    if (i < n) { key = items[i].key; tile = items[i].tile; }
    sk[j] = key;
    st[j] = tile;
  }
  int prev = kChunk;
  for (int k = 2; k <= kChunk; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      if (j > 64 || prev > 64) __syncthreads(); else wave_sync();
#pragma unroll
      for (int r = 0; r < kChunk / (2 * kChunkThreads); ++r) {
        const int q = r * kChunkThreads + threadIdx.x;
        const int i = ((q & ~(j - 1)) << 1) | (q & (j - 1));
        const uint64_t ka = sk[i], kb = sk[i + j];
        const uint32_t ta = st[i], tb = st[i + j];
        const bool b_first = kb < ka || (kb == ka && tb < ta);
        const bool sw = ((i & k) == 0) == b_first;  // ascending half: swap if b < a
        sk[i] = sw ? kb : ka;
        sk[i + j] = sw ? ka : kb;
        st[i] = sw ? tb : ta;
        st[i + j] = sw ? ta : tb;
      }
      prev = j;
    }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kChunk / kChunkThreads; ++r) {
    const int j = r * kChunkThreads + threadIdx.x;
    const int64_t i = base + j;
    if (i < n) {
      if (pack) {
        pack_record(pa, state, i, st[j]);
      } else {
        SortItem x;
        x.key = sk[j];
        x.tile = st[j];
        x.aux = 0u;  // the merge passes pack from the encoder outputs
        items[i] = x;
      }
    }
  }
}

// One multiway merge pass: runs of 2^logw sorted items, groups of F runs.
// An item's output slot is the first slot of its group, plus its index in its
// own run, plus, for every other run of the group, the number of that run's
// items that order before it.  That count is found digit by digit in radix
// 2^LOGR: each level probes 2^LOGR - 1 positions of every run, all loads
// independent and issued together (addresses clamped in range, results
// masked), so a level costs one memory round trip.  Wide groups use binary
// digits (F loads per level); the last pass over a few long runs uses base-8
// digits, which cuts the number of round trips by three.
template <int LOGR, int F>
__global__ __launch_bounds__(256) void k_merge_runs(const SortItem* __restrict__ in, uint64_t* state, int logw,
                                                    SortItem* __restrict__ out, int pack, PackArgs pa) {
  constexpr int NP = (1 << LOGR) - 1;  // probes per run per level
  const int64_t n = (int64_t)state[kSegK];
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const SortItem x = in[i];
  const int64_t w = (int64_t)1 << logw;
  const int64_t run = i >> logw;
  const int64_t g0 = run - run % F;
  int64_t len[F];
  int64_t cnt[F];
#pragma unroll
  for (int r = 0; r < F; ++r) {
    const int64_t rem = n - ((g0 + r) << logw);
    len[r] = (g0 + r == run || rem <= 0) ? 0 : (rem < w ? rem : w);
    cnt[r] = 0;
  }
  // largest power of 2^LOGR not above w: the count's top digit is then at most
  // w / top < 2^LOGR
  for (int64_t step = (int64_t)1 << (LOGR * (logw / LOGR)); step >= 1; step >>= LOGR) {
    SortItem y[F][NP];
#pragma unroll
    for (int r = 0; r < F; ++r) {
      const int64_t st = (g0 + r) << logw;
#pragma unroll
      for (int j = 1; j <= NP; ++j) {
        const int64_t probe = cnt[r] + j * step;
        y[r][j - 1] = in[len[r] > 0 ? st + (probe <= len[r] ? probe : len[r]) - 1 : i];
      }
    }
#pragma unroll
    for (int r = 0; r < F; ++r) {
      int c = 0;
#pragma unroll
      for (int j = 1; j <= NP; ++j) c += (int)((cnt[r] + j * step <= len[r]) & kv_less(y[r][j - 1], x));
      cnt[r] += c * step;
    }
  }
  int64_t pos = (g0 << logw) + (i - (run << logw));
#pragma unroll
  for (int r = 0; r < F; ++r) pos += cnt[r];
  if (pack) pack_record(pa, state, pos, x.tile);
  else out[pos] = x;
}

// ---------------------------------------------------------------- radix sort of large survivor sets
// Least-significant-digit radix sort on the 64-bit key, 8-bit digits, eight
// stable passes (the items enter in tile order, so equal keys keep
// increasing tiles, the same total order as the merge path).  A pass is a
// block histogram (kRsItems items per block), a scan per digit over the
// blocks, and a scatter in which every block first orders its items by digit
// in LDS (index order within a digit: within a wavefront by matching digits
// with ballots, across the block's four wavefronts and its rounds through LDS
// counters) and then writes them in that order, so that each digit's run of
// the block goes out as adjacent stores rather than one scattered 16-byte
// store per lane.  The last pass packs the records instead of writing items.
constexpr int kRsBits = 8;
constexpr int kRsBins = 1 << kRsBits;
constexpr int kRsThreads = 256;
constexpr int kRsRounds = 16;
constexpr int kRsItems = kRsThreads * kRsRounds;
constexpr int64_t kRadixMin = int64_t(1) << 20;  // record caps above this use the radix sort

__global__ __launch_bounds__(kRsThreads) void k_rs_hist(const SortItem* __restrict__ in, const uint64_t* state,
                                                        int shift, uint32_t* __restrict__ hist, int nblk) {
  __shared__ uint32_t h[kRsBins];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int64_t n = (int64_t)state[kSegK];
  const int64_t base = (int64_t)blockIdx.x * kRsItems;
  uint64_t keys[kRsRounds];  // every load issued before the first count
#pragma unroll
  for (int r = 0; r < kRsRounds; ++r) {
    const int64_t i = base + r * kRsThreads + threadIdx.x;
    keys[r] = i < n ? in[i].key : 0;
  }
#pragma unroll
  for (int r = 0; r < kRsRounds; ++r) {
    const int64_t i = base + r * kRsThreads + threadIdx.x;
    if (i < n) atomicAdd(&h[(uint32_t)(keys[r] >> shift) & (kRsBins - 1)], 1u);
  }
  __syncthreads();
  hist[(int64_t)threadIdx.x * nblk + blockIdx.x] = h[threadIdx.x];
}

// One block per digit: exclusive scan of the digit's counts over the blocks
// (in place), and the digit's total.
__global__ __launch_bounds__(1024) void k_rs_scan(uint32_t* __restrict__ hist, int nblk, uint32_t* __restrict__ tot) {
  __shared__ uint64_t s_wave[16];
  uint32_t* row = hist + (int64_t)blockIdx.x * nblk;
  uint64_t carry = 0;
  for (int c0 = 0; c0 < nblk; c0 += 1024) {
    const int i = c0 + threadIdx.x;
    const uint64_t v = i < nblk ? row[i] : 0;
    uint64_t t;
    const uint64_t incl = scan1024(v, s_wave, &t);
    if (i < nblk) row[i] = (uint32_t)(carry + incl - v);
    carry += t;
  }
  if (threadIdx.x == 0) tot[blockIdx.x] = (uint32_t)carry;
}

__global__ __launch_bounds__(kRsThreads) void k_rs_scatter(const SortItem* __restrict__ in, SortItem* __restrict__ out,
                                                           uint64_t* state, int shift,
                                                           const uint32_t* __restrict__ hist, int nblk,
                                                           const uint32_t* __restrict__ tot, int pack, PackArgs pa) {
  __shared__ uint32_t dbase[kRsBins];         // first slot of each digit for this block
  __shared__ uint32_t lstart[kRsBins];        // first place of each digit in the block's digit order
  __shared__ uint32_t lcur[kRsBins];          // next place of each digit in that order
  __shared__ uint32_t wc[kRsThreads / 64][kRsBins];  // items per digit of each wavefront in the round
  __shared__ uint64_t s_wave[kRsThreads / 64];
  __shared__ SortItem s_items[kRsItems];      // the block's items in digit order (stable within a digit)
  const int64_t n = (int64_t)state[kSegK];
  const int64_t base = (int64_t)blockIdx.x * kRsItems;
  if (base >= n) return;  // uniform per block
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  // exclusive scan of one value per digit (thread t holds digit t's) over the
  // block's 256 threads
  auto scan256 = [&](uint32_t v) -> uint32_t {
    uint32_t x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    if (lane == 63) s_wave[w] = x;
    __syncthreads();
    uint32_t before = 0;
#pragma unroll
    for (int k = 0; k < kRsThreads / 64; ++k) before += k < w ? (uint32_t)s_wave[k] : 0u;
    __syncthreads();  // s_wave is reused by the next scan
    return before + x - v;
  };
  // digit bases: exclusive scan of the 256 totals, plus this block's prefix
  dbase[t] = scan256(tot[t]) + hist[(int64_t)t * nblk + blockIdx.x];
  const uint64_t lt = lanemask_lt();
  // every round's item is loaded before the first round (one wait, not one
  // per round)
  SortItem xs[kRsRounds];
#pragma unroll
  for (int r = 0; r < kRsRounds; ++r) {
    const int64_t i = base + r * kRsThreads + t;
    xs[r].key = 0; xs[r].tile = 0; xs[r].aux = 0;
    if (i < n) xs[r] = in[i];
  }
  // the block's count of each digit, then where each digit's run starts in
  // the block's digit order
  lcur[t] = 0;
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kRsRounds; ++r)
    if (base + r * kRsThreads + t < n) atomicAdd(&lcur[(uint32_t)(xs[r].key >> shift) & (kRsBins - 1)], 1u);
  __syncthreads();
  const uint32_t ls = scan256(lcur[t]);
  lstart[t] = ls;
  lcur[t] = ls;
  // place every item in the block's digit order: within a wavefront by
  // matching digits with ballots, across the block's wavefronts and its
  // rounds through LDS counters (index order within a digit)
#pragma unroll
  for (int r = 0; r < kRsRounds; ++r) {
#pragma unroll
    for (int k = 0; k < kRsThreads / 64; ++k) wc[k][t] = 0;
    __syncthreads();
    const int64_t i = base + r * kRsThreads + t;
    const bool valid = i < n;
    const SortItem x = xs[r];
    const uint32_t d = (uint32_t)(x.key >> shift) & (kRsBins - 1);
    // lanes of this wavefront holding the same digit
    uint64_t same = __ballot(valid);
#pragma unroll
    for (int b = 0; b < kRsBits; ++b) {
      const uint64_t bal = __ballot((d >> b) & 1u);
      same &= ((d >> b) & 1u) ? bal : ~bal;
    }
    const uint32_t rank = (uint32_t)__popcll(same & lt);
    if (valid && rank == 0) wc[w][d] = (uint32_t)__popcll(same);
    __syncthreads();
    if (valid) {
      uint32_t lp = lcur[d] + rank;
#pragma unroll
      for (int k = 0; k < kRsThreads / 64; ++k) lp += k < w ? wc[k][d] : 0u;
      s_items[lp] = x;
    }
    __syncthreads();
    uint32_t add = 0;
#pragma unroll
    for (int k = 0; k < kRsThreads / 64; ++k) add += wc[k][t];
    lcur[t] += add;
  }
  __syncthreads();
  // write the block's items in digit order: consecutive threads take
  // consecutive items, so each digit's run goes out as adjacent stores
  const int64_t m = n - base < kRsItems ? n - base : kRsItems;
#pragma unroll 4
  for (int r = 0; r < kRsRounds; ++r) {
    const int j = r * kRsThreads + t;
    if (j < m) {
      const SortItem x = s_items[j];
      const uint32_t d = (uint32_t)(x.key >> shift) & (kRsBins - 1);
      const uint32_t off = dbase[d] + ((uint32_t)j - lstart[d]);
      if (pack) pack_record(pa, state, (int64_t)off, x.tile, x.aux);
      else out[off] = x;
    }
  }
}

// ---------------------------------------------------------------- workspace
size_t rank_ws_bytes(size_t n_tiles, size_t k_cap) {
  const size_t cap = k_cap ? k_cap : 1;
  const size_t max_blocks = (n_tiles + kItems - 1) / kItems + 1;
  const size_t rs_blocks = (cap + kRsItems - 1) / kRsItems;
  size_t b = 0;
  b += align_up(cap * sizeof(SortItem), 256) * 2;
  b += align_up((max_blocks + 1) * 8, 256) * 2;
  b += align_up((size_t)kStateWords * 8, 256);
  b += align_up(rs_blocks * kRsBins * 4, 256) + align_up(kRsBins * 4, 256);
  return b;
}

RankWs carve_rank(void* base, size_t n_tiles, size_t k_cap) {
  const size_t cap = k_cap ? k_cap : 1;
  const size_t max_blocks = (n_tiles + kItems - 1) / kItems + 1;
  char* p = static_cast<char*>(base);
  RankWs w;
  w.items_a = reinterpret_cast<SortItem*>(p); p += align_up(cap * sizeof(SortItem), 256);
  w.items_b = reinterpret_cast<SortItem*>(p); p += align_up(cap * sizeof(SortItem), 256);
  w.blk_a = reinterpret_cast<uint64_t*>(p); p += align_up((max_blocks + 1) * 8, 256);
  w.blk_b = reinterpret_cast<uint64_t*>(p); p += align_up((max_blocks + 1) * 8, 256);
  w.state = reinterpret_cast<uint64_t*>(p); p += align_up((size_t)kStateWords * 8, 256);
  w.rs_nblk = (cap + kRsItems - 1) / kRsItems;
  w.rs_hist = reinterpret_cast<uint32_t*>(p); p += align_up(w.rs_nblk * kRsBins * 4, 256);
  w.rs_tot = reinterpret_cast<uint32_t*>(p);
  w.cap = cap;
  w.max_blocks = max_blocks;
  return w;
}

hipError_t launch_rank_init(const RankWs& ws, hipStream_t st) {
  hipLaunchKernelGGL(k_rank_init, dim3(1), dim3(256), 0, st, ws.state);
  return hipGetLastError();
}

// One segment: count -> select -> compact -> sort -> pack, all on the device.
// `cap` bounds K (the budget's record count, at most n); grids are sized by it
// and kernels read the actual K from the state.
hipError_t launch_rank_segment(const double* gain, int64_t t0, int64_t n, int64_t cap, const RankWs& ws,
                               const uint16_t* seed, const int8_t* code, const uint16_t* scale, int P, int b,
                               int idx_bits, int seed_bits, int scale_bits, int L, uint64_t h,
                               uint64_t stream_cap, uint8_t* stream_out, hipStream_t st) {
  const double* g = gain + t0;
  int64_t cb = (n + kThreads - 1) / kThreads;
  if (cb > 512) cb = 512;
  if (cb < 1) cb = 1;
  hipLaunchKernelGGL(k_count_hist, dim3((unsigned)cb), dim3(kThreads), 0, st, g, n, ws.state);
  // passes 1..5 over the digits 12, 12, 12, 12 and 4 bits below the top one
  const int shifts[6] = {64 - kSelBits, 64 - 2 * kSelBits, 64 - 3 * kSelBits, 64 - 4 * kSelBits, 64 - 5 * kSelBits, 0};
  const int widths[6] = {kSelBits, kSelBits, kSelBits, kSelBits, kSelBits, 4};
  // fewer blocks than the counting pass: every block repeats the pick (a read
  // of the 32 KB histogram), and the keys under the prefix thin out fast
  int64_t sb = (n + 4 * kThreads - 1) / (4 * kThreads);
  if (sb > 128) sb = 128;
  if (sb < 1) sb = 1;
  for (int pass = 1; pass <= 5; ++pass)
    hipLaunchKernelGGL(k_select_pass, dim3((unsigned)sb), dim3(kThreads), 0, st, g, n, ws.state,
                       (int64_t)(cap > 0 ? cap : 0), pass, shifts[pass - 1], widths[pass - 1], shifts[pass],
                       widths[pass]);
  // the first compaction launch finishes the select and records the totals
  int64_t nbc = (n + kItems - 1) / kItems;
  if (nbc < 1) nbc = 1;
  hipLaunchKernelGGL(k_compact_count, dim3((unsigned)nbc), dim3(kThreads), 0, st, g, n, ws.state, ws.blk_a, ws.blk_b);
  hipLaunchKernelGGL(k_compact_scan, dim3(1), dim3(1024), 0, st, ws.blk_a, ws.blk_b, nbc, ws.state);
  if (cap <= 0 || n <= 0) return hipGetLastError();
  hipLaunchKernelGGL(k_compact_write, dim3((unsigned)nbc), dim3(kThreads), 0, st, g, seed, scale, t0, n, ws.state,
                     ws.blk_a, ws.blk_b, ws.items_a);
  // sort the survivors ascending on (~key, tile): LDS chunks, then multiway
  // merges; the final pass packs the records instead of writing items
  const PackArgs pa{seed, code, scale, P, b, idx_bits, seed_bits, scale_bits, L, h, stream_cap, stream_out};
  if (cap > kRadixMin) {
    const int nblk = (int)ws.rs_nblk;
    SortItem* in = ws.items_a;
    SortItem* out = ws.items_b;
    for (int pass = 0; pass < 64 / kRsBits; ++pass) {
      const int shift = pass * kRsBits;
      const int last = pass == 64 / kRsBits - 1 ? 1 : 0;
      hipLaunchKernelGGL(k_rs_hist, dim3((unsigned)nblk), dim3(kRsThreads), 0, st, in, ws.state, shift, ws.rs_hist,
                         nblk);
      hipLaunchKernelGGL(k_rs_scan, dim3(kRsBins), dim3(1024), 0, st, ws.rs_hist, nblk, ws.rs_tot);
      hipLaunchKernelGGL(k_rs_scatter, dim3((unsigned)nblk), dim3(kRsThreads), 0, st, in, out, ws.state, shift,
                         ws.rs_hist, nblk, ws.rs_tot, last, pa);
      SortItem* tt = in; in = out; out = tt;
    }
    return hipGetLastError();
  }
  int passes = 0;
  for (int logw = kLogChunk; ((int64_t)1 << logw) < cap; logw += cap <= ((int64_t)4 << logw) ? 2 : kLogFan) ++passes;
  hipLaunchKernelGGL(k_sort_chunks, dim3((unsigned)((cap + kChunk - 1) / kChunk)), dim3(kChunkThreads), 0, st,
                     ws.items_a, ws.state, passes == 0 ? 1 : 0, pa);
  SortItem* in = ws.items_a;
  SortItem* out = ws.items_b;
  int done = 0;
  for (int logw = kLogChunk; ((int64_t)1 << logw) < cap;) {
    const dim3 grid((unsigned)((cap + 255) / 256));
    const int last = ++done == passes ? 1 : 0;
    if (cap <= ((int64_t)4 << logw)) {  // at most four runs left: one base-8 pass
      hipLaunchKernelGGL((k_merge_runs<3, 4>), grid, dim3(256), 0, st, in, ws.state, logw, out, last, pa);
      logw += 2;
    } else {
      hipLaunchKernelGGL((k_merge_runs<1, kFan>), grid, dim3(256), 0, st, in, ws.state, logw, out, last, pa);
      logw += kLogFan;
    }
    SortItem* t = in; in = out; out = t;
  }
  return hipGetLastError();
}

// Totals of one call: records, eligible tiles, no-space flag.
const uint64_t* rank_totals(const RankWs& ws) { return ws.state + kTotK; }

}  // namespace awsrc
