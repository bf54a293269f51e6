// Internal declarations shared by the AWSRC HIP sources (not part of the ABI).
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/awsrc.h"

namespace awsrc {

constexpr int kMaxP = 16;        // basis columns per seed
constexpr int kMaxC = 128;       // tile length
constexpr int kTop = 2;          // screened candidates kept per tile for the fp64 re-score

// splitmix64 (Steele, Lea & Flood 2014): output n of the stream started at
// state `key`; the state advances by the golden-ratio increment before each
// output, which then passes through the variant-13 mixer.
__host__ __device__ __forceinline__ uint64_t splitmix64(uint64_t key, uint64_t n) {
  uint64_t z = key + (n + 1ull) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Device tables of the S seeded bases (generator version 1):
//   sign[s][w]      sign words, bit j%64 of word j/64 set <=> sigma_j = -1
//   mask[s][p][w]   bit j set <=> B_s[j, p] < 0, i.e. sigma_j xor parity(j & c_p)
//   col[s][p]       the P selected Hadamard columns (draw order)
//   tsign[s][j]     bit p set <=> B_s[j, p] < 0 (the mask transposed, one u16 per coordinate)
struct BasisTables {
  uint64_t* sign;
  uint64_t* mask;
  uint8_t* col;
  uint16_t* tsign;
  uint8_t* perm;   // [S][kMaxC] pi(j) (generator version 2)
  uint8_t* iperm;  // [S][kMaxC] pi^-1(i) (generator version 2)
};

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

inline size_t basis_bytes(int S, int P) {
  return align_up((size_t)S * 2 * 8, 256) + align_up((size_t)S * P * 2 * 8, 256) +
         align_up((size_t)S * kMaxP, 256) + align_up((size_t)S * kMaxC * 2, 256) +
         2 * align_up((size_t)S * kMaxC, 256);
}

inline BasisTables carve_basis(void* base, int S, int P) {
  char* p = static_cast<char*>(base);
  BasisTables t;
  t.sign = reinterpret_cast<uint64_t*>(p);
  p += align_up((size_t)S * 2 * 8, 256);
  t.mask = reinterpret_cast<uint64_t*>(p);
  p += align_up((size_t)S * P * 2 * 8, 256);
  t.col = reinterpret_cast<uint8_t*>(p);
  p += align_up((size_t)S * kMaxP, 256);
  t.tsign = reinterpret_cast<uint16_t*>(p);
  p += align_up((size_t)S * kMaxC * 2, 256);
  t.perm = reinterpret_cast<uint8_t*>(p);
  p += align_up((size_t)S * kMaxC, 256);
  t.iperm = reinterpret_cast<uint8_t*>(p);
  return t;
}

// Number of floats per (column block, seed) entry of the per-column factor
// table, G = B^T D B + eps I = L diag(e) L^T with L unit lower triangular:
// the strict lower part of L packed row by row (entry (p, k), k < p, at
// p (p - 1) / 2 + k), then 1 / e, then e.  Padded columns (p >= P) have
// L = 0 and e = 1.
inline int colfac_stride(int P) {
  int n = P * (P - 1) / 2 + 2 * P;
  return (n + 3) & ~3;
}


__host__ __device__ __forceinline__ int ltri(int p, int k) { return p * (p - 1) / 2 + k; }

// Knife edges of the fp32 screen.  The screen takes the rounding decisions of
// Sec. 3.2 (the scale, then every code) in fp32, the re-score in fp64 with
// the full chain; the two agree except where a decision lies within the
// screen's rounding error of its threshold, and there the screen scores a
// different rounding of the fit (by up to a few 1e-3 of the gain).  The
// screen flags such candidates (bit kEdge of a list entry's seed word) so
// that the re-score's window around them is the wide one below:
//   scale: m / qmax within 4e-6 (relative) of an fp16 rounding midpoint, or
//          of a power of two for the power-of-two format, or an fp16
//          subnormal scale;
//   codes: some |alpha_p / scale| < qmax within 1e-4 + 2e-5 |alpha_p / scale|
//          of a half-integer.
// The tolerances are some ten times the screen's relative error in alpha at
// the workloads' conditioning (measured: a few 1e-7).
constexpr uint32_t kEdge = 1u << 16;
__host__ __device__ __forceinline__ int list_seed(uint32_t w) { return (int)(w & 0xFFFFu); }

// The re-score's window below the best screened score g of a tile with
// weighted energy e = sum_j d_j r_j^2: a second kept seed is re-scored in
// fp64 when its screened score lies within it.  Narrow (1e-4 |g| + 1e-7 e)
// unless one of the two is flagged as a knife edge (3e-2 |g| + 3e-5 e, ten
// times the largest effect of a differing rounding seen).
__host__ __device__ __forceinline__ float rescore_window(float g, float e, bool edge) {
  return edge ? 3e-2f * fabsf(g) + 3e-5f * e : 1e-4f * fabsf(g) + 1e-7f * e;
}

// The screens' pruning threshold lowered by a relative 2^-9: a candidate is
// scored in full when its bound exceeds it.  The margin covers the fp32
// rounding of the bound and of the score (each a few ulps of the bound); it
// is applied to the threshold, which changes only in scoring rounds, rather
// than to every candidate's bound.
__device__ __forceinline__ float slack_thr(float thr) { return thr - fabsf(thr) * 0x1p-9f; }

__device__ __forceinline__ bool code_edge(float x, float qmax) {
  const float ax = fabsf(x);
  return ax < qmax && 0.5f - fabsf(x - rintf(x)) < 1e-4f + 2e-5f * ax;
}

// Screen-precision scale of max |alpha| = m: fp16 f16(m / qmax) with
// saturation, or the power of two 2^e, e = ceil(log2(m / qmax)), from the
// exponent and mantissa bits of the fp32 quotient.  The caller's values may
// be 2^RAW times the real ones (the unscaled projections of the matrix-core
// screens); the rounding is taken on the real value, as in the re-score.
// Returns the scale (in the caller's units), sets *isc to its reciprocal (0
// when the scale is 0) and *edge when the choice is on a knife edge (above).
// The format is a template argument: as a run-time flag it slowed the
// matrix-core screens by about a quarter.
template <bool POW2, int RAW = 0>
__device__ __forceinline__ float screen_scale(float m, float inv_qmax, float* isc, bool* edge) {
  const float x = m * inv_qmax * (1.0f / (float)(1 << RAW));  // real units, exact
  if constexpr (POW2) {
    const uint32_t xb = __float_as_uint(x);
    const uint32_t mb = xb & 0x7FFFFFu;
    int e = (int)((xb >> 23) & 0xFFu) - 127 + (mb ? 1 : 0);
    e = e < -126 ? -126 : (e > 127 - RAW ? 127 - RAW : e);
    *edge = x > 0.0f && (mb < 32u || mb > 0x7FFFFFu - 32u);
    *isc = x > 0.0f ? __uint_as_float((uint32_t)(127 - e - RAW) << 23) : 0.0f;
    return x > 0.0f ? __uint_as_float((uint32_t)(127 + e + RAW) << 23) : 0.0f;
  }
  uint16_t hb = __half_as_ushort(__float2half_rn(x));
  if ((hb & 0x7FFFu) == 0x7C00u) hb = 0x7BFFu;  // saturate at 65504
  const float sr = __half2float(__ushort_as_half(hb));
  // the rounding midpoints next to sr lie half an fp16 spacing away (below a
  // power of two the spacing underneath is half as wide)
  const uint32_t sb = __float_as_uint(sr);
  const int E = (int)((sb >> 23) & 0xFFu) - 127;
  float half = __uint_as_float((uint32_t)((E - 10 < -24 ? -24 : E - 10) - 1 + 127) << 23);
  if (x < sr && (sb & 0x7FFFFFu) == 0 && E > -14) half *= 0.5f;
  *edge = sr > 0.0f && (fabsf(fabsf(x - sr) - half) < 4e-6f * x || E < -14);
  const float sc = sr * (float)(1 << RAW);
  *isc = sc > 0.0f ? __builtin_amdgcn_rcpf(sc) : 0.0f;
  return sc;
}

// Screen score of one (tile, seed) from the per-column factor f (a table
// entry as above, read through any pointer type): solves G alpha = b with
// the LDL^T factor, quantizes alpha with one scale (screen_scale; POW2
// selects the power-of-two format), q = clamp(rint(alpha / scale)), and
// returns scale (2 q.b - scale q^T G q).  That is the exact gain
// 2 a.b - a^T G0 a of the quantized fit minus scale^2 eps |q|^2 (relative
// size ~ lambda), which the fp64 re-score of the kept seeds removes.  Uses
// q.b = (L^T q).w with w = L^-1 b, and q^T G q = sum_k e_k (L^T q)_k^2.
// *edge: a rounding decision on a knife edge (above).
//
// Split in two: screen_fwd solves L w = b and returns b^T G^-1 b =
// sum_k w_k^2 / e_k, the score of the unquantized optimum alpha = G^-1 b.
// The score is a concave quadratic in the coefficient vector c = scale q,
// 2 c.b - c^T G c, whose maximum over all c is that value, so no scale and
// codes can score above it: a candidate whose bound is below the score a
// tile already holds cannot enter its list.  screen_gain_w finishes the
// score from w.
template <int PB, typename FP>
__device__ __forceinline__ float screen_fwd(const float (&b)[PB], const FP& f, float (&w)[PB]) {
  constexpr int LS = PB * (PB - 1) / 2;
  float bound = 0.0f;
#pragma unroll
  for (int p = 0; p < PB; ++p) {
    float t = b[p];
#pragma unroll
    for (int k = 0; k < p; ++k) t = fmaf(-f[ltri(p, k)], w[k], t);
    w[p] = t;
    bound = fmaf(t * f[LS + p], t, bound);
  }
  return bound;
}

template <int PB, bool POW2, int RAW, typename FP>
__device__ __forceinline__ float screen_gain_w(const float (&w)[PB], const FP& f, float qmax, float inv_qmax,
                                               bool* edge) {
  constexpr int LS = PB * (PB - 1) / 2;
  float al[PB];
#pragma unroll
  for (int p = PB - 1; p >= 0; --p) {
    float t = w[p] * f[LS + p];
#pragma unroll
    for (int k = p + 1; k < PB; ++k) t = fmaf(-f[ltri(k, p)], al[k], t);
    al[p] = t;
  }
  float m = 0.0f;
#pragma unroll
  for (int p = 0; p < PB; ++p) m = fmaxf(m, fabsf(al[p]));
  float isc;
  bool ed;
  const float sc = screen_scale<POW2, RAW>(m, inv_qmax, &isc, &ed);
  float q[PB];
#pragma unroll
  for (int p = 0; p < PB; ++p) {
    const float x = al[p] * isc;
    q[p] = __builtin_amdgcn_fmed3f(rintf(x), -qmax, qmax);
    ed = ed || code_edge(x, qmax);
  }
  *edge = ed;
  float t1 = 0.0f, quad = 0.0f;
#pragma unroll
  for (int k = 0; k < PB; ++k) {
    float y = q[k];
#pragma unroll
    for (int i = k + 1; i < PB; ++i) y = fmaf(f[ltri(i, k)], q[i], y);
    t1 = fmaf(y, w[k], t1);
    quad = fmaf(f[LS + PB + k] * y, y, quad);
  }
  return sc * (2.0f * t1 - sc * quad);  // 0 when the scale is 0 (all codes 0)
}

template <int PB, bool POW2, int RAW, typename FP>
__device__ __forceinline__ float screen_score_ldl(const float (&b)[PB], const FP& f, float qmax, float inv_qmax,
                                                  bool* edge) {
  float w[PB];
  (void)screen_fwd<PB>(b, f, w);
  return screen_gain_w<PB, POW2, RAW>(w, f, qmax, inv_qmax, edge);
}

// ---------------------------------------------------------------- launchers
// Each returns hipSuccess or the first HIP error.
// Basis tables of GenBasis version gen_version (1: signs and columns; 2: also
// the seeded coordinate permutation, B_s[j, p] = sigma_j H[pi(j), c_p]/sqrt(C)).
hipError_t launch_gen_basis(uint64_t key, int C, int P, int S, int gen_version, BasisTables t, hipStream_t st);

// Scale double quantization of the backbone's group scales (blocks of 256).
int64_t sdq_blocks(int64_t n_groups);
hipError_t launch_sdq_encode(const uint16_t* s16, int64_t n_groups, int8_t* code, float* mean, float* step,
                             hipStream_t st);
hipError_t launch_sdq_dequant(const uint8_t* codes, const uint8_t* zero, const int8_t* sc, const float* mean,
                              const float* step, int64_t rows, int64_t cols, int group, float* W0, hipStream_t st);

hipError_t launch_backbone(const void* W, int w_dtype, int64_t rows, int64_t cols, int group,
                           uint8_t* codes, uint16_t* scale, uint8_t* zero, float* W0,
                           hipStream_t st);

struct EncodeArgs {
  const void* W;
  int w_dtype;
  const float* W0;
  const float* d;
  int d_mode;
  int64_t rows, cols;
  int C, P, b, S;
  double lambda;
  int scale_fmt;       // AWSRC_SCALE_FP16 or AWSRC_SCALE_POW2
  int gen_version;     // basis generator version (1 or 2)
  BasisTables basis;
  float* colfac;       // per-column factor table [nb][S][stride] (d_mode == PER_COL)
  double* wd64;        // per-column fp64 Walsh-Hadamard transform of d per block [nb][C]
  unsigned long long* scored;  // count of candidates scored in full (the pruned screen adds to it)
  void* frag;          // +-1 basis fragments of the matrix-core screen
  float* top_gain;     // [T][nsplit][kTop] screened gains per seed range, descending
                       // (the batched per-element encoder: [item][kTop][32], see launch_pe_lists_tile_order)
  uint32_t* top_seed;  // same layout: seed | kEdge flag
  int nsplit;          // seed ranges screened by separate waves (merged in the re-score)
  int fused_rescore;   // the screen also runs the re-score (no separate launch)
  uint16_t* seed_out;
  int8_t* code_out;
  uint16_t* scale_out;
  double* gain_out;
  float* alpha_out;
};

// One module of a batched encode: its inputs, shape, the global index of its
// first tile (outputs are concatenated in module order) and its first work
// item (32-row groups x column blocks, the same items for the screen and the
// re-score).
struct ModEntry {
  const void* W;
  const float* W0;
  const float* d;
  int64_t rows, cols;
  int64_t tile_off;
  int64_t item_off;
  int64_t pad_;  // keeps entries at 64 bytes
};
static_assert(sizeof(ModEntry) == 64, "module table entries are 64 bytes");

// The module holding work item `item`: the last m with item_off <= item
// (modules without work items share their successor's offset and are
// skipped).  Wavefront-uniform.
__device__ __forceinline__ int find_module(const ModEntry* mods, int n, int64_t item) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (mods[mid].item_off <= item) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Work item of workgroup b of a one-dimensional grid of n workgroups, such
// that each of the eight XCDs (which take workgroups round-robin, b mod 8)
// gets one contiguous range of items: neighbouring items (the next column
// blocks of the same rows) then share one L2, where their partial writes to
// the same lines merge.  A bijection on [0, n).
__device__ __forceinline__ int64_t xcd_item(int64_t b, int64_t n) {
  constexpr int kXcd = 8;
  const int64_t x = b % kXcd, k = b / kXcd;
  const int64_t base = n / kXcd, rem = n % kXcd;
  return x * base + (x < rem ? x : rem) + k;
}

// Module tables are written on the device from chunks passed by value (no
// host copy, so the encoder stays asynchronous).
constexpr int kModChunk = 48;
struct ModChunk {
  ModEntry e[kModChunk];
};
hipError_t launch_mod_table(const ModEntry* host, int n, ModEntry* dev, hipStream_t st);

// The batched per-element encoder (C = 64, P <= 8, generator version 1): the
// pruned screen over every module's 32-row groups, then the fp64 re-score.
constexpr int kPeRows = 32;
bool pe_batched_supported(int C, int P, int d_mode, int gen_version);
size_t pe_colsh_bytes(int S);
hipError_t launch_pe_screen(const EncodeArgs& a, const ModEntry* mods, int n_mods, int64_t items, const void* frag,
                            uint32_t* colsh, hipStream_t st);
hipError_t launch_finalize_pe_modules(const EncodeArgs& a, const ModEntry* mods, int n_mods, int64_t items,
                                      hipStream_t st);
// The batched screen's top lists ([item][kTop][32], work-item major) in tile
// order ([T][kTop]), for awsrc_encode_screen_lists.
hipError_t launch_pe_lists_tile_order(const float* tg, const uint32_t* ts, const ModEntry* mods, int n_mods,
                                      int64_t items, float* gain_out, uint32_t* seed_out, hipStream_t st);

bool encode_supported(int C, int P);
// the matrix-core screens: C = 64 (P <= 8), C = 128 (P <= 8, per-column
// weights); per-element weights need generator version 1 (XOR Gram gathers)
bool screen_mfma_supported(int C, int P, int d_mode, int gen_version);
int factor_pb(int C, int P);                 // padded P of the per-column factor table
size_t mfma_frag_bytes(int C, int S);
// +-1 bf16 basis fragments of the matrix-core screens, per seed pair and K step
hipError_t launch_mfma_frags(const BasisTables& bt, int C, int P, int S, void* frag, hipStream_t st);
// Seed ranges per tile for the screen (1 unless the matrix-core screen runs).
int screen_nsplit(int C, int P, int S, int64_t rows, int64_t cols, int d_mode, int gen_version);
hipError_t launch_encode_screen_mfma(const EncodeArgs& a, void* frag, hipStream_t st);
hipError_t launch_col_factors(const EncodeArgs& a, hipStream_t st);
hipError_t launch_encode_screen(const EncodeArgs& a, hipStream_t st);
hipError_t launch_encode_finalize(const EncodeArgs& a, hipStream_t st);
// Sets *a.scored to the count of candidates the screen will score in full
// without the pruned screen's help: 0 when it runs (it adds its own), else
// every candidate.
// With `add`, the count is added to the one already there (a batch of
// modules encoded one by one).
hipError_t launch_scored_init(const EncodeArgs& a, hipStream_t st, bool add = false);
hipError_t launch_scored_zero(unsigned long long* p, hipStream_t st);
bool screen_pruned(int C, int P, int d_mode, int gen_version);
// Whether the pruned screen runs the fp64 re-score itself (one seed range per
// tile, generator version 1).
bool screen_fuses_rescore(int C, int P, int d_mode, int gen_version, int nsplit);

// ---------------------------------------------------------------- ranking
// One survivor of the selection: ~(gain key), its global tile index, and
// the tile's seed | scale << 16 (carried by the radix sort so that packing
// gathers only the codes).
struct __attribute__((aligned(16))) SortItem {
  uint64_t key;
  uint32_t tile;
  uint32_t aux;
};

struct RankWs {
  SortItem* items_a;     // [cap] survivors (ping)
  SortItem* items_b;     // [cap] (pong)
  uint64_t* blk_a;       // [max_blocks + 1] per-block counts / offsets
  uint64_t* blk_b;       // [max_blocks + 1]
  uint64_t* state;       // [kStateWords] select state, counters, totals, histogram
  uint32_t* rs_hist;     // [256][rs_nblk] radix-sort digit counts per block (large record caps)
  uint32_t* rs_tot;      // [256] digit totals
  size_t rs_nblk;
  size_t cap;
  size_t max_blocks;
};
size_t rank_ws_bytes(size_t n_tiles, size_t k_cap);
RankWs carve_rank(void* base, size_t n_tiles, size_t k_cap);

constexpr int kStateWords = 32 + 3 * 4096;  // rank state: scalars, pick states, three select histograms
hipError_t launch_rank_init(const RankWs& ws, hipStream_t st);
// Top-K of one tile segment (K = min(cap, eligible), found on the device),
// ordered by (gain desc, tile asc), packed at the segment's first free record
// slot of the stream; no host synchronization.
hipError_t launch_rank_segment(const double* gain, int64_t t0, int64_t n, int64_t cap, const RankWs& ws,
                               const uint16_t* seed, const int8_t* code, const uint16_t* scale, int P, int b,
                               int idx_bits, int seed_bits, int scale_bits, int L, uint64_t h,
                               uint64_t stream_cap, uint8_t* stream_out, hipStream_t st);
// Device words after all segments: [0] records, [1] eligible tiles, [2] no-space flag.
const uint64_t* rank_totals(const RankWs& ws);

// ---------------------------------------------------------------- decoding
struct DecodeArgs {
  const uint8_t* recs;   // first record
  int64_t K;
  int C, P, b, S;
  int idx_bits, seed_bits, L_rec;
  uint64_t T_total;
  int n_modules;
  const uint64_t* mod_tile_off;  // [n_modules + 1]
  const int64_t* mod_cols;       // [n_modules]
  void* const* mod_ptr;          // [n_modules] device pointers
  int w0_dtype;
  int scale_fmt;                 // AWSRC_SCALE_FP16 or AWSRC_SCALE_POW2
  BasisTables basis;
  // [ceil(T_total / 32)][2]: bit i of word w marks a record for tile
  // 32 w + i; the second word of each pair holds the number of record tiles
  // before word w (filled for the dense reconstruction), so that one 8-byte
  // read gives a tile's rank
  uint32_t* bitmap;
  unsigned long long* errors;    // [1]
  // [K][2] decoded records written by validation: {tile within module,
  // module, seed | scale << 16, sum of codes}, then the P codes as int8 (zero
  // padded to 16)
  uint4* dec;
  uint4* dec_t;                  // [K + 1][2] the same records in tile order (reconstruction)
  uint32_t* bsum;                // [ceil(words / 4096)] scan scratch
};
hipError_t launch_decode_validate(const DecodeArgs& a, hipStream_t st);
hipError_t launch_decode_apply(const DecodeArgs& a, hipStream_t st);

// Stored backbone of each module for the bf16 reconstruction: device table
// of device pointers, codes [n] | scale [n] | zero [n] (layouts of
// awsrc_backbone_rtn), n = n_modules.
// Device table of backbone pointers, rows of n_modules entries: codes, scale
// (fp16, or the SDQ scale codes), zero points, the kMaxPrefixOutputs target
// rows, then (SDQ) the block means and steps.
struct BackboneTabs {
  const uint64_t* ptr;
  int gshift;  // log2 of the backbone group
  int sdq;     // scales are SDQ codes with per-block mean and step
};
constexpr int kMaxPrefixOutputs = 8;  // targets of one awsrc_reconstruct_bf16_prefixes call
constexpr int kBbRowSdqMean = 3 + kMaxPrefixOutputs;
constexpr int kBbRowSdqStep = 4 + kMaxPrefixOutputs;
constexpr int kBbRows = 5 + kMaxPrefixOutputs;
constexpr int kSdqBlock = 256;        // groups per SDQ block (mean and step)
// Dense bf16 reconstruction; toff is a host copy of the tile offsets (one
// launch per window of modules).  n_out == 0: into the plan's (bf16) module
// buffers with every record; else into n_out targets whose module pointer
// rows follow the backbone's in bb.ptr, target o with the records whose
// place in the stream is below K_out[o].
hipError_t launch_reconstruct_bf16(const DecodeArgs& a, const BackboneTabs& bb, const uint64_t* toff, int n_out,
                                   const uint32_t* K_out, hipStream_t st);

}  // namespace awsrc
