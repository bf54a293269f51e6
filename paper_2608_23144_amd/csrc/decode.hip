// Decoder (Sec. 3.2): every record regenerates its basis B_s and adds
// B_s (scale * q) onto its tile of W0; tiles without a record are untouched.
//
// validate - one thread per record: field ranges, finite non-negative scale,
//            and a bitmap over tiles that catches a tile appearing twice
//            (records of a valid stream touch disjoint tiles, which is what
//            lets the apply pass run without atomics or ordering);
// validate also writes each record in a decoded form (tile within its
//            module, module, seed, scale, codes and their sum);
// apply    - C/8 lanes per record, eight consecutive weights per lane; each
//            weight gets rhat_j = (1/sqrt(C)) sum_p (+-1) scale*q_p with the
//            signs of row j of B_s read from the transposed sign table;
// reconstruct (dense bf16) - the decoded records put in tile order (prefix
//            counts of the bitmap words give each record tile its rank), then
//            one streaming pass over every weight.
#include <type_traits>

#include "awsrc_internal.h"

namespace awsrc {

constexpr int kLdsModules = 256;  // module tables up to this size are staged in LDS

typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_a8_t __attribute__((ext_vector_type(4), aligned(8)));  // 8-byte aligned

#define HIP_RETURN_IF(expr)            \
  do {                                 \
    const hipError_t e_ = (expr);      \
    if (e_ != hipSuccess) return e_;   \
  } while (0)

struct Rec {
  uint64_t idx;
  uint32_t seed;
  int32_t q[kMaxP];
  uint32_t scale;
};

__device__ __forceinline__ uint64_t get_bits(const uint64_t (&w)[3], int& pos, int nbits) {
  if (nbits <= 0) return 0;
  const int o = pos & 63, k = pos >> 6;
  uint64_t v = w[k] >> o;
  if (o + nbits > 64) v |= w[k + 1] << (64 - o);
  pos += nbits;
  return nbits == 64 ? v : (v & ((1ull << nbits) - 1ull));
}

// Record i of the stream, read with aligned 4-byte loads.  The record area
// starts h = 40 + 8n bytes into an 8-byte aligned stream, so it is 4-byte
// aligned.  A record of at most 32 + 16 + 16*8 + 16 = 192 bits (24 bytes)
// spans at most 7 words from its first word; records whose 7 words all lie
// in the record area load them unconditionally (independent loads in flight
// together), the last few records take a guarded byte-wise path.
__device__ __forceinline__ Rec parse(const DecodeArgs& a, int64_t i) {
  const int64_t o = i * a.L_rec;
  const int64_t total = a.K * a.L_rec;
  const int64_t d0 = o >> 2;
  const int sh = (int)(o & 3) * 8;
  const uint32_t* r32 = reinterpret_cast<const uint32_t*>(a.recs);
  uint32_t wd[7];
  if (d0 + 7 <= (total >> 2)) {
#pragma unroll
    for (int k = 0; k < 7; ++k) wd[k] = r32[d0 + k];
  } else {
#pragma unroll
    for (int k = 0; k < 7; ++k) {
      uint32_t v = 0;
      for (int b = 0; b < 4; ++b) {
        const int64_t at = (d0 + k) * 4 + b;
        if (at < o + a.L_rec && at < total) v |= (uint32_t)a.recs[at] << (8 * b);
      }
      wd[k] = v;
    }
  }
  uint64_t w[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const uint64_t lo = (uint64_t)wd[2 * k] | ((uint64_t)wd[2 * k + 1] << 32);
    const uint64_t hi = (uint64_t)wd[2 * k + 2];
    w[k] = sh ? ((lo >> sh) | (hi << (64 - sh))) : lo;
  }
  // bits beyond the record are not used: every field lies within L_rec bytes
  Rec out;
  int pos = 0;
  out.idx = get_bits(w, pos, a.idx_bits);
  out.seed = (uint32_t)get_bits(w, pos, a.seed_bits);
  // loops over the fixed maximum with a guard keep every index static (a
  // loop bounded by P would put the codes in scratch memory)
#pragma unroll
  for (int p = 0; p < kMaxP; ++p) {
    int64_t c = 0;
    if (p < a.P) {
      c = (int64_t)get_bits(w, pos, a.b);
      if (c >> (a.b - 1)) c -= (int64_t)1 << a.b;
    }
    out.q[p] = (int32_t)c;
  }
  out.scale = (uint32_t)get_bits(w, pos, a.scale_fmt == AWSRC_SCALE_POW2 ? 8 : 16);
  return out;
}

__global__ void k_fill_u32(uint32_t* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// field checks of one record (everything but a repeated tile)
__device__ __forceinline__ bool record_fields_ok(const DecodeArgs& a, const Rec& r) {
  const int qmax = (1 << (a.b - 1)) - 1;
  bool bad = r.idx >= a.T_total || r.seed >= (uint32_t)a.S;
#pragma unroll
  for (int p = 0; p < kMaxP; ++p) bad |= p < a.P && (r.q[p] < -qmax || r.q[p] > qmax);
  // fp16 scale: negative, inf or NaN; every 8-bit exponent is valid
  if (a.scale_fmt != AWSRC_SCALE_POW2) bad |= (r.scale & 0x8000u) != 0 || (r.scale & 0x7C00u) == 0x7C00u;
  return !bad;
}

// The module table (tile offsets) is staged in LDS when it has at most
// kLdsModules + 1 entries, so that each record's binary search for its module
// reads no global memory.
__global__ __launch_bounds__(256) void k_decode_validate(DecodeArgs a) {
  __shared__ uint64_t s_off[kLdsModules + 1];
  const bool lds_tab = a.n_modules <= kLdsModules;
  if (lds_tab)
    for (int m = threadIdx.x; m <= a.n_modules; m += blockDim.x) s_off[m] = a.mod_tile_off[m];
  __syncthreads();
  const uint64_t* toff = lds_tab ? s_off : a.mod_tile_off;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.K) return;
  const Rec r = parse(a, i);
  bool bad = !record_fields_ok(a, r);
  if (!bad) {
    const uint32_t bit = 1u << (r.idx & 31);
    const uint32_t old = atomicOr(&a.bitmap[2 * (r.idx >> 5)], bit);
    bad = (old & bit) != 0;
  }
  if (bad) atomicAdd(a.errors, 1ull);
  // decoded form for the apply pass (only used once the whole stream is valid)
  int lo = 0, hi = a.n_modules - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (toff[mid] <= r.idx) lo = mid; else hi = mid - 1;
  }
  uint32_t qw[4] = {0u, 0u, 0u, 0u};
  int32_t tot = 0;
#pragma unroll
  for (int p = 0; p < kMaxP; ++p) {
    if (p >= a.P) continue;
    qw[p >> 2] |= ((uint32_t)r.q[p] & 0xFFu) << (8 * (p & 3));
    tot += r.q[p];
  }
  a.dec[2 * i] = make_uint4((uint32_t)(r.idx - toff[lo]), (uint32_t)lo, r.seed | (r.scale << 16),
                            (uint32_t)tot);
  a.dec[2 * i + 1] = make_uint4(qw[0], qw[1], qw[2], qw[3]);
}

// ---------------------------------------------------------------- bitmap prefix counts
constexpr int kScanWords = 16;                    // bitmap words per thread
constexpr int kScanThreads = 256;
constexpr int kScanBlockWords = kScanWords * kScanThreads;

// exclusive scan over the NT threads of a block; *total gets the block sum
template <int NT>
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* s_wave, uint32_t* total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_wave[wv] = x;
  __syncthreads();
  uint32_t before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) {
    const uint32_t t = s_wave[w];
    before += w < wv ? t : 0u;
    tot += t;
  }
  __syncthreads();
  *total = tot;
  return before + x - v;
}

__device__ __forceinline__ uint32_t thread_word_count(const uint32_t* bitmap, int64_t nw, int64_t w0) {
  uint32_t c = 0;
#pragma unroll
  for (int k = 0; k < kScanWords; ++k)
    if (w0 + k < nw) c += __popc(bitmap[2 * (w0 + k)]);
  return c;
}

__global__ __launch_bounds__(kScanThreads) void k_scan_sums(DecodeArgs a, int64_t nw) {
  __shared__ uint32_t s_wave[kScanThreads / 64];
  const int64_t w0 = (int64_t)blockIdx.x * kScanBlockWords + (int64_t)threadIdx.x * kScanWords;
  uint32_t tot;
  block_exclusive_scan<kScanThreads>(thread_word_count(a.bitmap, nw, w0), s_wave, &tot);
  if (threadIdx.x == 0) a.bsum[blockIdx.x] = tot;
}

// one block: exclusive scan of the per-block sums, in place
__global__ __launch_bounds__(1024) void k_scan_top(DecodeArgs a, int64_t nb) {
  __shared__ uint32_t s_wave[16];
  uint32_t carry = 0;
  for (int64_t i0 = 0; i0 < nb; i0 += 1024) {
    const int64_t i = i0 + threadIdx.x;
    const uint32_t v = i < nb ? a.bsum[i] : 0u;
    uint32_t tot;
    const uint32_t ex = block_exclusive_scan<1024>(v, s_wave, &tot);
    if (i < nb) a.bsum[i] = carry + ex;
    carry += tot;
  }
}

__global__ __launch_bounds__(kScanThreads) void k_scan_words(DecodeArgs a, int64_t nw) {
  __shared__ uint32_t s_wave[kScanThreads / 64];
  const int64_t w0 = (int64_t)blockIdx.x * kScanBlockWords + (int64_t)threadIdx.x * kScanWords;
  uint32_t tot;
  uint32_t run = a.bsum[blockIdx.x] +
                 block_exclusive_scan<kScanThreads>(thread_word_count(a.bitmap, nw, w0), s_wave, &tot);
#pragma unroll
  for (int k = 0; k < kScanWords; ++k) {
    if (w0 + k < nw) {
      const uint32_t word = a.bitmap[2 * (w0 + k)];
      a.bitmap[2 * (w0 + k) + 1] = run;
      run += __popc(word);
    }
  }
}

// rank of record tile t among all record tiles (tile order)
__device__ __forceinline__ uint32_t tile_rank(const DecodeArgs& a, uint64_t t) {
  const u32x2_t wp = *reinterpret_cast<const u32x2_t*>(a.bitmap + 2 * (t >> 5));
  return wp.y + __popc(wp.x & ((1u << (t & 31)) - 1u));
}

// decoded record i (stream order) copied to its tile-order rank
__global__ __launch_bounds__(256) void k_decode_tile_order(DecodeArgs a) {
  __shared__ uint64_t s_off[kLdsModules];  // module tile offsets (first kLdsModules)
  const bool lds_tab = a.n_modules <= kLdsModules;
  if (lds_tab)
    for (int m = threadIdx.x; m < a.n_modules; m += blockDim.x) s_off[m] = a.mod_tile_off[m];
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.K) return;
  const uint4 e0 = a.dec[2 * i];
  const uint4 e1 = a.dec[2 * i + 1];
  const uint32_t k = tile_rank(a, (lds_tab ? s_off[e0.y] : a.mod_tile_off[e0.y]) + e0.x);
  // the tile-ordered copy carries the record's place in the stream in its
  // first word (the tile is implied by the position), for the nested-prefix
  // reconstruction
  a.dec_t[2 * (size_t)k] = make_uint4((uint32_t)i, e0.y, e0.z, e0.w);
  a.dec_t[2 * (size_t)k + 1] = e1;
}

// C/8 lanes per record, eight consecutive weights per lane.  With integer
// codes, C * rhat_j / sqrt(C) = scale * sum_p sign_jp q_p is scale times an
// exact integer: sum_p q_p minus twice the codes at the negative entries of
// row j, the latter one int8 dot product per four codes against a 0/1 byte
// mask spread from the row's sign bits.  Blocks loop over record groups so
// that the table of W0 pointers is staged in LDS once per block.
template <int C, typename TW, int G>
__global__ __launch_bounds__(256) void k_decode_apply(DecodeArgs a) {
  constexpr int LPR = C / 8;           // lanes per record
  constexpr int RPB = 256 / LPR;       // records per block per iteration
  __shared__ void* s_ptr[kLdsModules];
  const bool lds_tab = a.n_modules <= kLdsModules;
  if (lds_tab)
    for (int m = threadIdx.x; m < a.n_modules; m += 256) s_ptr[m] = a.mod_ptr[m];
  __syncthreads();
  void* const* mptr = lds_tab ? s_ptr : a.mod_ptr;
  constexpr float isq = (C == 16) ? 0.25f : (C == 32) ? 0.17677669529663688f
                      : (C == 64) ? 0.125f : 0.08838834764831845f;
  const int sub = threadIdx.x % LPR;
  for (int64_t i = (int64_t)blockIdx.x * RPB + threadIdx.x / LPR; i < a.K; i += (int64_t)gridDim.x * RPB) {
    const uint4 e0 = a.dec[2 * i];
    const uint4 e1 = a.dec[2 * i + 1];
    const uint32_t q4[4] = {e1.x, e1.y, e1.z, e1.w};
    // signs of this lane's eight rows of B_s, one u16 of P bits per row: rows
    // 8 sub .. 8 sub + 7 (bf16 targets), or rows 4 sub .. 4 sub + 3 of each
    // half of the tile (fp32 targets, so that the 16-byte accesses of the
    // record's lanes are adjacent)
    const uint16_t* trow = a.basis.tsign + (size_t)(e0.z & 0xFFFFu) * kMaxC;
    uint32_t tw[4];
    if constexpr (sizeof(TW) == 4) {
      const uint2 t0 = *reinterpret_cast<const uint2*>(trow + sub * 4);
      const uint2 t1 = *reinterpret_cast<const uint2*>(trow + C / 2 + sub * 4);
      tw[0] = t0.x; tw[1] = t0.y; tw[2] = t1.x; tw[3] = t1.y;
    } else {
      const uint4 tsv = *reinterpret_cast<const uint4*>(trow + sub * 8);
      tw[0] = tsv.x; tw[1] = tsv.y; tw[2] = tsv.z; tw[3] = tsv.w;
    }
    const uint32_t sfield = e0.z >> 16;
    const float scl = a.scale_fmt == AWSRC_SCALE_POW2 ? ldexpf(isq, (int)sfield - 128)
                                                      : __half2float(__ushort_as_half((uint16_t)sfield)) * isq;
    const int32_t tot = (int32_t)e0.w;
    float add[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t ts = (tw[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
      int32_t neg = 0;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const uint32_t mask = (((ts >> (4 * g)) & 0xFu) * 0x204081u) & 0x01010101u;
        neg = __builtin_amdgcn_sdot4((int)mask, (int)q4[g], neg, false);
      }
      add[e] = (float)(tot - 2 * neg) * scl;
    }
    TW* W0 = static_cast<TW*>(mptr[e0.y]);
    if constexpr (sizeof(TW) == 4) {
      float4* q0 = reinterpret_cast<float4*>(W0 + (int64_t)e0.x * C + sub * 4);
      float4* q1 = q0 + C / 8;  // the same place in the tile's second half
      float4 v0 = *q0, v1 = *q1;
      v0.x += add[0]; v0.y += add[1]; v0.z += add[2]; v0.w += add[3];
      v1.x += add[4]; v1.y += add[5]; v1.z += add[6]; v1.w += add[7];
      *q0 = v0;
      *q1 = v1;
    } else {
      uint4* q = reinterpret_cast<uint4*>(W0 + (int64_t)e0.x * C + sub * 8);
      const uint4 v = *q;
      const uint32_t in[4] = {v.x, v.y, v.z, v.w};
      uint32_t o[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        uint32_t h2 = 0;
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const uint32_t bits = e ? (in[k] & 0xFFFF0000u) : (in[k] << 16);
          uint32_t u = __float_as_uint(__uint_as_float(bits) + add[2 * k + e]);
          u += 0x7FFFu + ((u >> 16) & 1u);  // round to nearest even (finite values)
          h2 |= (u >> 16) << (16 * e);
        }
        o[k] = h2;
      }
      *q = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
}

// ---------------------------------------------------------------- dense bf16 reconstruction
// One streaming pass over every weight of every module.  Lanes own units of
// UW consecutive weights (UW / 2 bytes of codes in, 2 UW bytes of
// bf16 out, consecutive lanes on consecutive units), W0 =
// f32(q - z) * s recomputed from the backbone.  A lane whose tile has a record
// (bit set in the validation bitmap) reads it at the tile's rank in the
// tile-ordered decoded records (a coalesced read: neighbouring lanes' records
// are neighbours) and adds its corrections before the single rounding to
// bf16.  The sign table sits in LDS when it fits.
//
// The loop is software-pipelined over the block's chunks so that no wait on
// a load also waits on the stores just issued (loads and stores share one
// in-order counter): in the iteration that computes chunk c it issues the
// backbone loads of chunk c + step, the bitmap words of chunk c + 2 step and
// the decoded records of chunk c + step (whose bitmap words arrived one
// iteration earlier), and only then computes and stores chunk c.

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t bf16_pair(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));  // nearest even
}

// global-address-space views: loads and stores through them are issued as
// global (not flat) memory instructions
#define AWSRC_GLOBAL __attribute__((address_space(1)))

constexpr int kRecThreads = 512;
// Weights per unit of a pass with NO targets.  Four targets: 8, so that a
// unit's 16 output bytes per target are one store and consecutive lanes'
// stores are adjacent (a wavefront's store covers 1 KB without gaps); with 16
// (two 16-byte stores per lane and target, 32 bytes apart) the address and
// data units of the CUs, not memory, bounded the pass (busy 99% of its
// cycles), and it ran 20% slower.  One target: 16, which halves the loads per
// weight where stores are fewer (4-7% faster at C = 128, even at C = 64).
template <int NO>
constexpr int rec_unit_w() { return NO == 1 ? 16 : 8; }
constexpr int kRecUnits = 2;                 // units per lane per chunk
constexpr int kTsignLdsMax = 64 * 1024;      // sign tables up to this size are staged in LDS
// the codes of one unit of UW weights: UW / 2 bytes
template <int UW>
using UnitCodes = typename std::conditional<UW == 16, u32x2_t, uint32_t>::type;

__device__ __forceinline__ uint32_t code_word(const u32x2_t& q, int i) { return q[i]; }
__device__ __forceinline__ uint32_t code_word(const uint32_t& q, int) { return q; }

template <int NU, int UW>
struct RecBackbone {                         // backbone words of one chunk
  UnitCodes<UW> q[NU];
  uint32_t s[NU], z[NU];                     // fp16 scale bits, or the SDQ scale code (sign-extended)
  float mu[NU], st[NU];                      // SDQ: the mean and step of the scale code's block
  uint32_t m[NU];                            // module (within the window) and first element of the unit
  uint64_t el[NU];
  bool ok[NU];
};
template <int NU>
struct RecBits {                             // bitmap word and its prefix count per unit
  uint32_t word[NU], pre[NU];
};
template <int NU, int G>
struct RecDec {                              // decoded record per unit (record 0 when none)
  u32x2_t sw[NU];                            // seed | scale << 16, sum of codes
  // the codes, four per word; only the words in use are loaded, so that no
  // dead part of a load destination is ever reused while the load is in flight
  typename std::conditional<(G <= 2), u32x2_t, u32x4_t>::type q[NU];
  uint32_t rank[NU];                         // the record's place in the stream (nested prefixes)
  bool rec[NU];
};

// Outputs of one reconstruction launch: NO bf16 targets whose module pointer
// rows follow the backbone's in the staged table (rows 3 + o0 ..); with
// `ranked`, a record goes into output o only when its place in the stream is
// below K[o] (nested prefixes of one stream), else into every output (the
// plan's own targets, rows of mod_ptr).
struct RecOut {
  uint32_t K[4];
  int o0;
  int ranked;
};

// One launch covers a window of at most kLdsModules consecutive modules,
// whose table rows (tile offset, codes, scale, zero and output pointers) are
// staged in LDS, so that the per-lane module walk never waits on the
// vector-memory counter.  Unit uw of a module covers its elements
// [16 uw, 16 uw + 16) (rows are whole multiples of the group, hence of 16),
// and its backbone group is element / group.  Every load is issued unconditionally (units
// past the window end are clamped to its last unit and not stored).
template <int C, int G, bool TS_LDS, int NO, bool SDQ>
__global__ __launch_bounds__(kRecThreads) void k_reconstruct(DecodeArgs a, BackboneTabs bb, RecOut ro, int m0,
                                                             int nm) {
  constexpr int NT = kRecThreads, NU = kRecUnits;
  constexpr int kUnitW = rec_unit_w<NO>();               // weights per unit
  constexpr int kLogUnitW = kUnitW == 16 ? 4 : 3;
  constexpr int UPT = C / kUnitW;                        // lanes per tile
  constexpr int LOG_UPT = ((C == 16) ? 4 : (C == 32) ? 5 : (C == 64) ? 6 : 7) - kLogUnitW;
  constexpr float isq = (C == 16) ? 0.25f : (C == 32) ? 0.17677669529663688f
                      : (C == 64) ? 0.125f : 0.08838834764831845f;
  extern __shared__ __align__(16) uint64_t s_dyn[];
  // LDS: [tile offsets nm+1 | codes nm | scale nm | zero nm | out NO x nm
  // | SDQ: block means nm | block steps nm] then [S][C] sign rows
  constexpr int NROW = 4 + NO + (SDQ ? 2 : 0);
  uint64_t* s_off = s_dyn;
  uint64_t* s_cp = s_off + nm + 1;
  uint64_t* s_sp = s_cp + nm;
  uint64_t* s_zp = s_sp + nm;
  uint64_t* s_op = s_zp + nm;
  uint64_t* s_mp = s_op + NO * nm;
  uint64_t* s_tp = s_mp + nm;
  uint16_t* s_ts = reinterpret_cast<uint16_t*>(s_dyn + ((NROW * nm + 1 + 1) & ~1));
  const uint32_t n_all = (uint32_t)a.n_modules;
  for (int i = threadIdx.x; i <= nm; i += NT) s_off[i] = a.mod_tile_off[m0 + i];
  for (int i = threadIdx.x; i < nm; i += NT) {
    s_cp[i] = bb.ptr[m0 + i];
    s_sp[i] = bb.ptr[n_all + m0 + i];
    s_zp[i] = bb.ptr[2 * n_all + m0 + i];
#pragma unroll
    for (int o = 0; o < NO; ++o)
      s_op[o * nm + i] = ro.ranked ? bb.ptr[(3 + ro.o0 + o) * (size_t)n_all + m0 + i]
                                   : reinterpret_cast<uint64_t>(a.mod_ptr[m0 + i]);
    if constexpr (SDQ) {
      s_mp[i] = bb.ptr[(size_t)kBbRowSdqMean * n_all + m0 + i];
      s_tp[i] = bb.ptr[(size_t)kBbRowSdqStep * n_all + m0 + i];
    }
  }
  if constexpr (TS_LDS) {
    constexpr int PER_SEED = C / 8;                      // 16-byte pieces per seed
    for (int i = threadIdx.x; i < a.S * PER_SEED; i += NT) {
      const int sd = i / PER_SEED, j = i - sd * PER_SEED;
      reinterpret_cast<uint4*>(s_ts)[i] = reinterpret_cast<const uint4*>(a.basis.tsign + (size_t)sd * kMaxC)[j];
    }
  }
  __syncthreads();
  const uint64_t u_begin = s_off[0] << LOG_UPT, u_end = s_off[nm] << LOG_UPT;
  const uint64_t CH = (uint64_t)NU * NT;
  const uint64_t step = (uint64_t)gridDim.x * CH;
  const uint64_t c0 = u_begin + (uint64_t)blockIdx.x * CH;

  // per-lane module state for the backbone loads; their units only move
  // forward, so the walk costs at most nm steps per lane per launch
  int m = 0;
  uint64_t m_lo = u_begin, m_hi = s_off[1] << LOG_UPT;

  auto issue_backbone = [&](uint64_t c, RecBackbone<NU, kUnitW>& B) {
#pragma unroll
    for (int k = 0; k < NU; ++k) {
      uint64_t u = c + (uint64_t)(k * NT) + threadIdx.x;
      B.ok[k] = u < u_end;
      u = B.ok[k] ? u : u_end - 1;
      if (u >= m_hi) {
        do { ++m; } while ((s_off[m + 1] << LOG_UPT) <= u);
        m_lo = s_off[m] << LOG_UPT;
        m_hi = s_off[m + 1] << LOG_UPT;
      }
      const uint64_t el = (u - m_lo) << kLogUnitW;       // first element of the unit
      const uint64_t g = el >> bb.gshift;
      B.q[k] = *((const AWSRC_GLOBAL UnitCodes<kUnitW>*)s_cp[m] + (el >> kLogUnitW));
      if constexpr (SDQ) {
        B.s[k] = (uint32_t)(int32_t)((const AWSRC_GLOBAL int8_t*)s_sp[m])[g];
        B.mu[k] = ((const AWSRC_GLOBAL float*)s_mp[m])[g / kSdqBlock];
        B.st[k] = ((const AWSRC_GLOBAL float*)s_tp[m])[g / kSdqBlock];
      } else {
        B.s[k] = ((const AWSRC_GLOBAL uint16_t*)s_sp[m])[g];
      }
      B.z[k] = ((const AWSRC_GLOBAL uint8_t*)s_zp[m])[g];
      B.m[k] = (uint32_t)m;
      B.el[k] = el;
    }
  };
  auto issue_bits = [&](uint64_t c, RecBits<NU>& W) {
#pragma unroll
    for (int k = 0; k < NU; ++k) {
      uint64_t u = c + (uint64_t)(k * NT) + threadIdx.x;
      u = u < u_end ? u : u_end - 1;
      const uint64_t w = u >> (LOG_UPT + 5);
      const u32x2_t wp = *reinterpret_cast<const u32x2_t*>(a.bitmap + 2 * w);
      W.word[k] = wp.x;
      W.pre[k] = wp.y;
    }
  };
  auto issue_dec = [&](uint64_t c, const RecBits<NU>& W, RecDec<NU, G>& D) {
#pragma unroll
    for (int k = 0; k < NU; ++k) {
      const uint64_t u = c + (uint64_t)(k * NT) + threadIdx.x;
      const uint32_t sh = (uint32_t)(u >> LOG_UPT) & 31u;
      D.rec[k] = (W.word[k] >> sh) & 1u;
      const uint32_t r = D.rec[k] ? W.pre[k] + __popc(W.word[k] & ((1u << sh) - 1u)) : 0u;
      const uint32_t* dp = reinterpret_cast<const uint32_t*>(a.dec_t) + 8 * (size_t)r;
      D.rank[k] = ro.ranked ? dp[0] : 0u;
      if constexpr (G <= 2) {
        // words 2..5 (seed | scale, sum of codes, the two code words) in one load
        const u32x4_a8_t v = *reinterpret_cast<const u32x4_a8_t*>(dp + 2);
        D.sw[k] = u32x2_t{v[0], v[1]};
        D.q[k] = u32x2_t{v[2], v[3]};
      } else {
        D.sw[k] = *reinterpret_cast<const u32x2_t*>(dp + 2);
        D.q[k] = *reinterpret_cast<const u32x4_t*>(dp + 4);
      }
    }
  };
  auto compute = [&](uint64_t c, const RecBackbone<NU, kUnitW>& B, const RecDec<NU, G>& D) {
#pragma unroll
    for (int k = 0; k < NU; ++k) {
      if (!B.ok[k]) continue;
      const uint64_t u = c + (uint64_t)(k * NT) + threadIdx.x;
      // the group's scale: fp16, or the SDQ scale f32(mu + code step) (both
      // terms and their sum exact in fp64, so one rounding)
      float s;
      if constexpr (SDQ)
        s = (float)((double)B.mu[k] + (double)(int32_t)B.s[k] * (double)B.st[k]);
      else
        s = __half2float(__ushort_as_half((uint16_t)B.s[k]));
      const float z = (float)B.z[k];
      float w[kUnitW];
#pragma unroll
      for (int e = 0; e < kUnitW; ++e)
        w[e] = ((float)((code_word(B.q[k], e >> 3) >> (4 * (e & 7))) & 0xFu) - z) * s;
      float wr[kUnitW];
#pragma unroll
      for (int e = 0; e < kUnitW; ++e) wr[e] = w[e];
      if (D.rec[k]) {
        // rows sub*kUnitW .. of B_s: sqrt(C) rhat_j = scale (sum_p q_p - 2 sum
        // of the codes at the negative entries of row j)
        const int sub = (int)(u & (UPT - 1));
        const uint32_t sd = D.sw[k].x & 0xFFFFu;
        const uint4* trow;
        if constexpr (TS_LDS)
          trow = reinterpret_cast<const uint4*>(s_ts + (size_t)sd * C + sub * kUnitW);
        else
          trow = reinterpret_cast<const uint4*>(a.basis.tsign + (size_t)sd * kMaxC + sub * kUnitW);
        uint32_t tw[kUnitW / 2];
#pragma unroll
        for (int i = 0; i < kUnitW / 8; ++i) {
          const uint4 t4 = trow[i];
          tw[4 * i] = t4.x; tw[4 * i + 1] = t4.y; tw[4 * i + 2] = t4.z; tw[4 * i + 3] = t4.w;
        }
        uint32_t q4[4] = {D.q[k][0], D.q[k][1], 0u, 0u};
        if constexpr (G > 2) {
          q4[2] = D.q[k][2];
          q4[3] = D.q[k][3];
        }
        const uint32_t sfield = D.sw[k].x >> 16;
        const float scl = a.scale_fmt == AWSRC_SCALE_POW2 ? ldexpf(isq, (int)sfield - 128)
                                                          : __half2float(__ushort_as_half((uint16_t)sfield)) * isq;
        const int32_t tot = (int32_t)D.sw[k].y;
#pragma unroll
        for (int e = 0; e < kUnitW; ++e) {
          const uint32_t ts = (tw[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
          int32_t neg = 0;
#pragma unroll
          for (int gg = 0; gg < G; ++gg) {
            const uint32_t mask = (((ts >> (4 * gg)) & 0xFu) * 0x204081u) & 0x01010101u;
            neg = __builtin_amdgcn_sdot4((int)mask, (int)q4[gg], neg, false);
          }
          wr[e] = w[e] + (float)(tot - 2 * neg) * scl;
        }
      }
      // the unit rounded with and (when it has a record) without the
      // correction; each output takes one of the two
      u32x4_t ob[kUnitW / 8], orc[kUnitW / 8];
#pragma unroll
      for (int i = 0; i < kUnitW / 8; ++i) {
        orc[i] = u32x4_t{bf16_pair(wr[8 * i], wr[8 * i + 1]), bf16_pair(wr[8 * i + 2], wr[8 * i + 3]),
                         bf16_pair(wr[8 * i + 4], wr[8 * i + 5]), bf16_pair(wr[8 * i + 6], wr[8 * i + 7])};
        if (ro.ranked)
          ob[i] = u32x4_t{bf16_pair(w[8 * i], w[8 * i + 1]), bf16_pair(w[8 * i + 2], w[8 * i + 3]),
                          bf16_pair(w[8 * i + 4], w[8 * i + 5]), bf16_pair(w[8 * i + 6], w[8 * i + 7])};
        else
          ob[i] = orc[i];
      }
#pragma unroll
      for (int o = 0; o < NO; ++o) {
        const bool with = !ro.ranked || (D.rec[k] && D.rank[k] < ro.K[o]);
        AWSRC_GLOBAL u32x4_t* out = (AWSRC_GLOBAL u32x4_t*)s_op[o * nm + B.m[k]] + (B.el[k] >> 3);
#pragma unroll
        for (int i = 0; i < kUnitW / 8; ++i) {
          // a select per word (a select of the whole arrays went through scratch)
          u32x4_t v;
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = with ? orc[i][j] : ob[i][j];
          out[i] = v;
        }
      }
    }
  };

  // two alternating register sets for the backbone words and the records,
  // so that nothing in flight is ever copied; the bitmap words of chunk
  // c + step are consumed (record loads) before the words of c + 2 step are
  // loaded into the same registers
  RecBackbone<NU, kUnitW> B0, B1;
  RecBits<NU> W;
  RecDec<NU, G> D0, D1;
  issue_bits(c0, W);
  issue_backbone(c0, B0);
  issue_dec(c0, W, D0);
  issue_bits(c0 + step, W);
  for (uint64_t c = c0; c < u_end; c += 2 * step) {
    issue_backbone(c + step, B1);
    issue_dec(c + step, W, D1);
    issue_bits(c + 2 * step, W);
    compute(c, B0, D0);
    if (c + step >= u_end) break;
    issue_backbone(c + 2 * step, B0);
    issue_dec(c + 2 * step, W, D0);
    issue_bits(c + 3 * step, W);
    compute(c + step, B1, D1);
  }
}

// dynamic LDS of one launch: module window table (rounded to 16 bytes) and
// the sign rows when staged
static size_t rec_lds_bytes(int C, int S, int nm, bool ts_lds, int no, bool sdq) {
  return (size_t)(((4 + no + (sdq ? 2 : 0)) * nm + 1 + 1) & ~1) * 8 + (ts_lds ? (size_t)S * C * 2 : 0);
}

// module windows: 256 modules for one output, 255 for four, so that two
// blocks still fit per CU with a 64 KB sign table staged: (4 + NO) x 8 bytes
// per module plus 16, and the sign rows, within half of the 160 KB
template <int NO, bool SDQ>
constexpr int rec_window() { return SDQ ? (NO == 1 ? kLdsModules : 200) : (NO == 1 ? kLdsModules : 255); }
static_assert(2 * (((4 + 4) * 255 + 2) * 8 + kTsignLdsMax) <= 160 * 1024, "two blocks per CU");
static_assert(2 * (((4 + 4 + 2) * 200 + 2) * 8 + kTsignLdsMax) <= 160 * 1024, "two blocks per CU (SDQ)");
static_assert(2 * (((4 + 1 + 2) * kLdsModules + 2) * 8 + kTsignLdsMax) <= 160 * 1024, "two blocks per CU (SDQ)");

template <int C, int G, bool TS_LDS, int NO, bool SDQ>
static hipError_t launch_rec_cgt(const DecodeArgs& a, const BackboneTabs& bb, const RecOut& ro, const uint64_t* toff,
                                 hipStream_t st) {
  constexpr int WIN = rec_window<NO, SDQ>();
  for (int m0 = 0; m0 < a.n_modules; m0 += WIN) {
    const int nm = a.n_modules - m0 < WIN ? a.n_modules - m0 : WIN;
    const size_t lds = rec_lds_bytes(C, a.S, nm, TS_LDS, NO, SDQ);
    int per_cu = 0;
    HIP_RETURN_IF(
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_reconstruct<C, G, TS_LDS, NO, SDQ>, kRecThreads, lds));
    if (per_cu < 1) per_cu = 1;
    const uint64_t units = (toff[m0 + nm] - toff[m0]) * (uint64_t)(C / rec_unit_w<NO>());
    const uint64_t chunks = (units + kRecUnits * kRecThreads - 1) / (kRecUnits * kRecThreads);
    // four times the blocks that fit at once, grid-stride beyond (more blocks
    // than resident keep the CUs full to the end: 2.5% faster on the 2.8G-
    // weight stack than resident blocks alone, no better at 16 times)
    uint64_t nb = (uint64_t)per_cu * 256 * 4;
    if (nb > chunks) nb = chunks;
    if (nb < 1) continue;
    hipLaunchKernelGGL((k_reconstruct<C, G, TS_LDS, NO, SDQ>), dim3((unsigned)nb), dim3(kRecThreads), lds, st, a, bb,
                       ro, m0, nm);
    HIP_RETURN_IF(hipGetLastError());
  }
  return hipSuccess;
}

template <int C, int G, int NO, bool SDQ>
static hipError_t launch_rec_cgn(const DecodeArgs& a, const BackboneTabs& bb, const RecOut& ro, const uint64_t* toff,
                                 hipStream_t st) {
  if ((size_t)a.S * C * 2 <= (size_t)kTsignLdsMax) return launch_rec_cgt<C, G, true, NO, SDQ>(a, bb, ro, toff, st);
  return launch_rec_cgt<C, G, false, NO, SDQ>(a, bb, ro, toff, st);
}

template <int C, int NO, bool SDQ>
static hipError_t launch_rec_cns(const DecodeArgs& a, const BackboneTabs& bb, const RecOut& ro, const uint64_t* toff,
                                 hipStream_t st) {
  switch ((a.P + 3) / 4) {
    case 1: return launch_rec_cgn<C, 1, NO, SDQ>(a, bb, ro, toff, st);
    case 2: return launch_rec_cgn<C, 2, NO, SDQ>(a, bb, ro, toff, st);
    case 3: return launch_rec_cgn<C, 3, NO, SDQ>(a, bb, ro, toff, st);
    default: return launch_rec_cgn<C, 4, NO, SDQ>(a, bb, ro, toff, st);
  }
}

template <int C, int NO>
static hipError_t launch_rec_cn(const DecodeArgs& a, const BackboneTabs& bb, const RecOut& ro, const uint64_t* toff,
                                hipStream_t st) {
  return bb.sdq ? launch_rec_cns<C, NO, true>(a, bb, ro, toff, st) : launch_rec_cns<C, NO, false>(a, bb, ro, toff, st);
}

// One pass: no == 1, or no == 4 (C >= 64 only).
static hipError_t launch_rec_pass(const DecodeArgs& a, const BackboneTabs& bb, const RecOut& ro, int no,
                                  const uint64_t* toff, hipStream_t st) {
  switch (a.C) {
    case 16: return launch_rec_cn<16, 1>(a, bb, ro, toff, st);
    case 32: return launch_rec_cn<32, 1>(a, bb, ro, toff, st);
    case 64: return no == 4 ? launch_rec_cn<64, 4>(a, bb, ro, toff, st) : launch_rec_cn<64, 1>(a, bb, ro, toff, st);
    case 128: return no == 4 ? launch_rec_cn<128, 4>(a, bb, ro, toff, st) : launch_rec_cn<128, 1>(a, bb, ro, toff, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_reconstruct_bf16(const DecodeArgs& a, const BackboneTabs& bb, const uint64_t* toff, int n_out,
                                   const uint32_t* K_out, hipStream_t st) {
  if (a.K > 0) {
    // the records in tile order: prefix counts of the bitmap words, then each
    // decoded record copied to its rank
    const int64_t nwords = (int64_t)((a.T_total + 31) / 32);
    const int64_t nb = (nwords + kScanBlockWords - 1) / kScanBlockWords;
    hipLaunchKernelGGL(k_scan_sums, dim3((unsigned)nb), dim3(kScanThreads), 0, st, a, nwords);
    hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(1024), 0, st, a, nb);
    hipLaunchKernelGGL(k_scan_words, dim3((unsigned)nb), dim3(kScanThreads), 0, st, a, nwords);
    hipLaunchKernelGGL(k_decode_tile_order, dim3((unsigned)((a.K + 255) / 256)), dim3(256), 0, st, a);
    HIP_RETURN_IF(hipGetLastError());
  }
  if (n_out == 0) {  // the plan's own targets, every record
    RecOut ro{};
    return launch_rec_pass(a, bb, ro, 1, toff, st);
  }
  for (int o0 = 0; o0 < n_out;) {
    const int no = (a.C >= 64 && n_out - o0 >= 4) ? 4 : 1;
    RecOut ro{};
    ro.ranked = 1;
    ro.o0 = o0;
    for (int o = 0; o < no; ++o) ro.K[o] = K_out[o0 + o];
    HIP_RETURN_IF(launch_rec_pass(a, bb, ro, no, toff, st));
    o0 += no;
  }
  return hipSuccess;
}

hipError_t launch_decode_validate(const DecodeArgs& a, hipStream_t st) {
  const int64_t nwords = (int64_t)((a.T_total + 31) / 32);
  int64_t fb = (nwords + 255) / 256;
  if (fb > 4096) fb = 4096;
  if (fb < 1) fb = 1;
  hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)fb), dim3(256), 0, st, a.bitmap, 2 * nwords);
  hipLaunchKernelGGL(k_fill_u32, dim3(1), dim3(64), 0, st, reinterpret_cast<uint32_t*>(a.errors), (int64_t)2);
  if (a.K > 0)
    hipLaunchKernelGGL(k_decode_validate, dim3((unsigned)((a.K + 255) / 256)), dim3(256), 0, st, a);
  return hipGetLastError();
}

template <int C, int G>
static hipError_t apply_cg(const DecodeArgs& a, hipStream_t st) {
  constexpr int RPB = 256 / (C / 8);
  // at most 64 blocks per CU, each looping over record groups (more blocks
  // than fit at once keep the CUs full to the end: a cap of 8 per CU measured
  // 3% slower on a 9.2M-record stream; one block per record group would
  // stage the module table once per group)
  int64_t nb = (a.K + RPB - 1) / RPB;
  if (nb > 256 * 64) nb = 256 * 64;
  const unsigned blocks = (unsigned)nb;
  if (a.w0_dtype == AWSRC_DTYPE_F32)
    hipLaunchKernelGGL((k_decode_apply<C, float, G>), dim3(blocks), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((k_decode_apply<C, uint16_t, G>), dim3(blocks), dim3(256), 0, st, a);
  return hipGetLastError();
}

template <int C>
static hipError_t apply_c(const DecodeArgs& a, hipStream_t st) {
  switch ((a.P + 3) / 4) {  // groups of four codes
    case 1: return apply_cg<C, 1>(a, st);
    case 2: return apply_cg<C, 2>(a, st);
    case 3: return apply_cg<C, 3>(a, st);
    default: return apply_cg<C, 4>(a, st);
  }
}

hipError_t launch_decode_apply(const DecodeArgs& a, hipStream_t st) {
  if (a.K <= 0) return hipSuccess;
  switch (a.C) {
    case 16: return apply_c<16>(a, st);
    case 32: return apply_c<32>(a, st);
    case 64: return apply_c<64>(a, st);
    case 128: return apply_c<128>(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace awsrc
