// extern "C" entry points of libawsrc: argument validation, workspace layout
// and kernel orchestration.  Every step of the codec itself runs in the HIP
// kernels of basis.hip, backbone.hip, encode*.hip, rank.hip and decode.hip.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <string>
#include <vector>

#include "awsrc_internal.h"

using namespace awsrc;

namespace {

thread_local std::string g_err;

awsrc_status fail(awsrc_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define HIPCHK(expr)                                                                   \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess) return fail(AWSRC_EDEVICE, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

int ceil_log2_u64(uint64_t n) {
  int b = 0;
  while (b < 64 && (1ull << b) < n) ++b;
  return b;
}

bool pow2_c(int C) { return C == 16 || C == 32 || C == 64 || C == 128; }

awsrc_status check_params(const awsrc_params* p) {
  if (!p) return fail(AWSRC_EINVAL, "params is NULL");
  if (!pow2_c(p->C)) return fail(AWSRC_EINVAL, "C=%d: must be 16, 32, 64 or 128", p->C);
  if (p->P < 1 || p->P > kMaxP || p->P > p->C) return fail(AWSRC_EINVAL, "P=%d out of range 1..min(C,16)", p->P);
  if (p->b < 2 || p->b > 8) return fail(AWSRC_EINVAL, "b=%d out of range 2..8", p->b);
  if (p->S < 2 || p->S > 65536) return fail(AWSRC_EINVAL, "S=%d out of range 2..65536", p->S);
  if (p->scale_fmt != AWSRC_SCALE_FP16 && p->scale_fmt != AWSRC_SCALE_POW2)
    return fail(AWSRC_EINVAL, "scale_fmt=%d unsupported", p->scale_fmt);
  if (p->idx_bits < 0 || p->idx_bits > 32) return fail(AWSRC_EINVAL, "idx_bits=%d out of range 0..32", p->idx_bits);
  if (p->gen_version != 1 && p->gen_version != 2) return fail(AWSRC_EINVAL, "gen_version=%d unsupported", p->gen_version);
  if (p->reserved != 0) return fail(AWSRC_EINVAL, "reserved field must be 0");
  if (!(p->ridge_lambda >= 0.0) || !isfinite(p->ridge_lambda)) return fail(AWSRC_EINVAL, "ridge_lambda must be finite and >= 0");
  return AWSRC_OK;
}

int index_bits(const awsrc_params* p, uint64_t T_total) {
  return p->idx_bits ? p->idx_bits : ceil_log2_u64(T_total);
}

int scale_field_bits(int scale_fmt) { return scale_fmt == AWSRC_SCALE_POW2 ? 8 : 16; }

int64_t rec_bytes(int ib, int S, int P, int b, int scale_bits) {
  return (ib + ceil_log2_u64((uint64_t)S) + P * b + scale_bits + 7) / 8;
}

void put_le(std::vector<uint8_t>& v, uint64_t x, int n) {
  for (int i = 0; i < n; ++i) v.push_back((uint8_t)(x >> (8 * i)));
}
uint64_t get_le(const uint8_t* p, int n) {
  uint64_t x = 0;
  for (int i = 0; i < n; ++i) x |= (uint64_t)p[i] << (8 * i);
  return x;
}

constexpr int kHeaderFixed = 40;

}  // namespace

extern "C" int32_t awsrc_abi_version(void) { return AWSRC_ABI_VERSION; }
extern "C" const char* awsrc_last_error(void) { return g_err.c_str(); }

extern "C" int64_t awsrc_record_bytes(const awsrc_params* p, int64_t T_total) {
  if (check_params(p) != AWSRC_OK || T_total < 1) return -1;
  return rec_bytes(index_bits(p, (uint64_t)T_total), p->S, p->P, p->b, scale_field_bits(p->scale_fmt));
}

extern "C" int64_t awsrc_header_bytes(int32_t n_modules) {
  return n_modules < 1 ? -1 : kHeaderFixed + 8 * (int64_t)n_modules;
}

extern "C" int64_t awsrc_budget_bytes(double bpw, int64_t n_weights) {
  if (!(bpw >= 0.0) || !isfinite(bpw) || n_weights < 0) return -1;
  return (int64_t)floor((bpw * (double)n_weights) / 8.0);
}

extern "C" int64_t awsrc_prefix_K(int64_t budget_bytes, int64_t h, int64_t L_rec, int64_t n_eligible) {
  if (h < 0 || L_rec < 1 || n_eligible < 0) return -1;
  if (budget_bytes < h) return AWSRC_ENOSPC;
  const int64_t k = (budget_bytes - h) / L_rec;
  return k < n_eligible ? k : n_eligible;
}

// ---------------------------------------------------------------- backbone
extern "C" awsrc_status awsrc_backbone_rtn(const void* W, int32_t w_dtype, int64_t rows, int64_t cols,
                                           int32_t group, uint8_t* codes, uint16_t* scale_f16,
                                           uint8_t* zero, float* W0_or_null, void* stream) {
  if (w_dtype != AWSRC_DTYPE_F32 && w_dtype != AWSRC_DTYPE_BF16) return fail(AWSRC_EINVAL, "bad w_dtype %d", w_dtype);
  if (group != 64 && group != 128 && group != 256) return fail(AWSRC_EINVAL, "group=%d: must be 64, 128 or 256", group);
  if (rows < 0 || cols < 1 || cols % group) return fail(AWSRC_EINVAL, "cols=%lld must be a positive multiple of group", (long long)cols);
  if (rows == 0) return AWSRC_OK;
  if (!W || !codes || !scale_f16 || !zero) return fail(AWSRC_EINVAL, "NULL buffer");
  if ((reinterpret_cast<uintptr_t>(W) | reinterpret_cast<uintptr_t>(W0_or_null)) & 15 ||
      reinterpret_cast<uintptr_t>(codes) & 3)
    return fail(AWSRC_EINVAL, "W and W0 must be 16-byte aligned, codes 4-byte aligned");
  HIPCHK(launch_backbone(W, w_dtype, rows, cols, group, codes, scale_f16, zero, W0_or_null,
                         (hipStream_t)stream));
  return AWSRC_OK;
}

// ---------------------------------------------------------------- encode
namespace {

// Workspace of one module on the per-module kernels (every path but the
// batched per-element one): size only, or carve it and launch.
size_t module_ws_bytes(const awsrc_params* p, int64_t rows, int64_t cols, int32_t d_mode) {
  const int64_t nb = cols / p->C;
  const int64_t T = rows * nb;
  const int PB = factor_pb(p->C, p->P);
  const size_t b_basis = align_up(basis_bytes(p->S, p->P), 256);
  const size_t b_fac = d_mode == AWSRC_D_PER_COL ? align_up((size_t)nb * p->S * colfac_stride(PB) * 4, 256) : 0;
  const size_t b_wd = d_mode == AWSRC_D_PER_COL ? align_up((size_t)nb * p->C * 8, 256) : 0;
  const size_t b_frag =
      screen_mfma_supported(p->C, p->P, d_mode, p->gen_version) ? align_up(mfma_frag_bytes(p->C, p->S), 256) : 0;
  const int nsplit = screen_nsplit(p->C, p->P, p->S, rows, cols, d_mode, p->gen_version);
  const size_t b_tg = align_up((size_t)T * nsplit * kTop * 4, 256);
  const size_t b_ts = align_up((size_t)T * nsplit * kTop * 4, 256);
  return 256 + b_basis + b_fac + b_wd + b_frag + b_tg + b_ts + 256;
}

awsrc_status encode_module(const awsrc_params* p, const void* W, int32_t w_dtype, const float* W0, int64_t rows,
                           int64_t cols, const float* d, int32_t d_mode, uint16_t* seed_out, int8_t* code_out,
                           uint16_t* scale_out, double* gain_out, float* alpha_or_null, char* ws, bool add_scored,
                           hipStream_t s) {
  const int64_t nb = cols / p->C;
  const int64_t T = rows * nb;
  const int PB = factor_pb(p->C, p->P);
  const size_t b_basis = align_up(basis_bytes(p->S, p->P), 256);
  const size_t b_fac = d_mode == AWSRC_D_PER_COL ? align_up((size_t)nb * p->S * colfac_stride(PB) * 4, 256) : 0;
  const size_t b_wd = d_mode == AWSRC_D_PER_COL ? align_up((size_t)nb * p->C * 8, 256) : 0;
  const size_t b_frag =
      screen_mfma_supported(p->C, p->P, d_mode, p->gen_version) ? align_up(mfma_frag_bytes(p->C, p->S), 256) : 0;
  const int nsplit = screen_nsplit(p->C, p->P, p->S, rows, cols, d_mode, p->gen_version);
  const size_t b_tg = align_up((size_t)T * nsplit * kTop * 4, 256);
  EncodeArgs a{};
  a.W = W; a.w_dtype = w_dtype; a.W0 = W0; a.d = d; a.d_mode = d_mode;
  a.rows = rows; a.cols = cols; a.C = p->C; a.P = p->P; a.b = p->b; a.S = p->S;
  a.lambda = p->ridge_lambda;
  a.scale_fmt = p->scale_fmt;
  a.gen_version = p->gen_version;
  a.scored = reinterpret_cast<unsigned long long*>(ws);
  ws += 256;
  a.basis = carve_basis(ws, p->S, p->P);
  ws += b_basis;
  a.colfac = b_fac ? reinterpret_cast<float*>(ws) : nullptr;
  ws += b_fac;
  a.wd64 = b_wd ? reinterpret_cast<double*>(ws) : nullptr;
  ws += b_wd;
  a.frag = b_frag ? static_cast<void*>(ws) : nullptr;
  ws += b_frag;
  a.top_gain = reinterpret_cast<float*>(ws);
  ws += b_tg;
  a.top_seed = reinterpret_cast<uint32_t*>(ws);
  a.nsplit = nsplit;
  a.fused_rescore = screen_fuses_rescore(p->C, p->P, d_mode, p->gen_version, nsplit) ? 1 : 0;
  a.seed_out = seed_out; a.code_out = code_out; a.scale_out = scale_out; a.gain_out = gain_out;
  a.alpha_out = alpha_or_null;
  HIPCHK(launch_scored_init(a, s, add_scored));
  HIPCHK(launch_gen_basis(p->basis_key, p->C, p->P, p->S, p->gen_version, a.basis, s));
  if (d_mode == AWSRC_D_PER_COL) HIPCHK(launch_col_factors(a, s));
  HIPCHK(launch_encode_screen(a, s));
  if (!a.fused_rescore) HIPCHK(launch_encode_finalize(a, s));
  return AWSRC_OK;
}

// Workspace of the batched per-element encoder: count | basis | fragments |
// shifted columns | module table | top lists of every work item (32 tiles
// each, padded where a module's rows end mid-group).
struct PeLayout {
  size_t basis, frag, colsh, mods, tg, ts, total;
};
int64_t pe_items(const awsrc_params* p, int n_modules, const int64_t* rows, const int64_t* cols) {
  int64_t items = 0;
  for (int m = 0; m < n_modules; ++m) items += (rows[m] + kPeRows - 1) / kPeRows * (cols[m] / p->C);
  return items;
}
PeLayout pe_layout(const awsrc_params* p, int n_modules, int64_t items) {
  PeLayout l;
  l.basis = align_up(basis_bytes(p->S, p->P), 256);
  l.frag = align_up(mfma_frag_bytes(p->C, p->S), 256);
  l.colsh = align_up(pe_colsh_bytes(p->S), 256);
  l.mods = align_up((size_t)n_modules * sizeof(ModEntry), 256);
  l.tg = align_up((size_t)items * kPeRows * kTop * 4, 256);
  l.ts = align_up((size_t)items * kPeRows * kTop * 4, 256);
  l.total = 256 + l.basis + l.frag + l.colsh + l.mods + l.tg + l.ts + 256;
  return l;
}

// The encoder over n modules with outputs concatenated in module order.
awsrc_status encode_modules(const awsrc_params* p, int32_t n_modules, const void* const* W, int32_t w_dtype,
                            const float* const* W0, const float* const* d, int32_t d_mode, const int64_t* rows,
                            const int64_t* cols, uint16_t* seed_out, int8_t* code_out, uint16_t* scale_out,
                            double* gain_out, float* alpha_or_null, void* workspace, size_t* ws_bytes, void* stream) {
  awsrc_status st = check_params(p);
  if (st) return st;
  if (!ws_bytes) return fail(AWSRC_EINVAL, "ws_bytes is NULL");
  if (w_dtype != AWSRC_DTYPE_F32 && w_dtype != AWSRC_DTYPE_BF16) return fail(AWSRC_EINVAL, "bad w_dtype %d", w_dtype);
  if (d_mode != AWSRC_D_PER_COL && d_mode != AWSRC_D_PER_ELEM) return fail(AWSRC_EINVAL, "bad d_mode %d", d_mode);
  if (!encode_supported(p->C, p->P)) return fail(AWSRC_EINVAL, "unsupported (C, P)");
  if (n_modules < 1 || !rows || !cols) return fail(AWSRC_EINVAL, "bad module table");
  int64_t T_total = 0;
  for (int m = 0; m < n_modules; ++m) {
    if (rows[m] < 0 || cols[m] < 1 || cols[m] % p->C)
      return fail(AWSRC_EINVAL, "module %d: cols=%lld must be a positive multiple of C=%d", m, (long long)cols[m], p->C);
    const int64_t T = rows[m] * (cols[m] / p->C);
    if (T > (int64_t)UINT32_MAX) return fail(AWSRC_EINVAL, "too many tiles in module %d", m);
    T_total += T;
  }
  if (T_total > (int64_t)UINT32_MAX) return fail(AWSRC_EINVAL, "more than 2^32 tiles");
  const bool batched = pe_batched_supported(p->C, p->P, d_mode, p->gen_version);
  size_t need = 0;
  if (batched) {
    need = pe_layout(p, n_modules, pe_items(p, n_modules, rows, cols)).total;
  } else {
    for (int m = 0; m < n_modules; ++m) {
      const size_t b = module_ws_bytes(p, rows[m], cols[m], d_mode);
      need = b > need ? b : need;
    }
  }
  if (!workspace) { *ws_bytes = need; return AWSRC_OK; }
  if (*ws_bytes < need) return fail(AWSRC_ENOSPC, "workspace %zu < %zu bytes", *ws_bytes, need);
  if (T_total == 0) return AWSRC_OK;
  if (!W || !W0 || !d || !seed_out || !code_out || !scale_out || !gain_out) return fail(AWSRC_EINVAL, "NULL buffer");
  for (int m = 0; m < n_modules; ++m) {
    if (rows[m] == 0) continue;
    if (!W[m] || !W0[m] || !d[m]) return fail(AWSRC_EINVAL, "NULL input of module %d", m);
    if ((reinterpret_cast<uintptr_t>(W[m]) | reinterpret_cast<uintptr_t>(W0[m]) | reinterpret_cast<uintptr_t>(d[m])) &
        15)
      return fail(AWSRC_EINVAL, "W, W0 and d must be 16-byte aligned (module %d)", m);
  }
  char* ws = reinterpret_cast<char*>(align_up(reinterpret_cast<uintptr_t>(workspace), 256));
  hipStream_t s = (hipStream_t)stream;
  if (!batched) {
    int64_t t0 = 0;
    bool first = true;
    for (int m = 0; m < n_modules; ++m) {
      const int64_t T = rows[m] * (cols[m] / p->C);
      if (T == 0) continue;
      st = encode_module(p, W[m], w_dtype, W0[m], rows[m], cols[m], d[m], d_mode, seed_out + t0,
                         code_out + t0 * p->P, scale_out + t0, gain_out + t0,
                         alpha_or_null ? alpha_or_null + t0 * p->P : nullptr, ws, !first, s);
      if (st) return st;
      first = false;
      t0 += T;
    }
    return AWSRC_OK;
  }
  const PeLayout l = pe_layout(p, n_modules, pe_items(p, n_modules, rows, cols));
  EncodeArgs a{};
  a.w_dtype = w_dtype; a.d_mode = d_mode;
  a.C = p->C; a.P = p->P; a.b = p->b; a.S = p->S;
  a.lambda = p->ridge_lambda;
  a.scale_fmt = p->scale_fmt;
  a.gen_version = p->gen_version;
  a.scored = reinterpret_cast<unsigned long long*>(ws);
  char* q = ws + 256;
  a.basis = carve_basis(q, p->S, p->P);
  q += l.basis;
  a.frag = q;
  q += l.frag;
  uint32_t* colsh = reinterpret_cast<uint32_t*>(q);
  q += l.colsh;
  ModEntry* mods = reinterpret_cast<ModEntry*>(q);
  q += l.mods;
  a.top_gain = reinterpret_cast<float*>(q);
  q += l.tg;
  a.top_seed = reinterpret_cast<uint32_t*>(q);
  a.nsplit = 1;
  a.seed_out = seed_out; a.code_out = code_out; a.scale_out = scale_out; a.gain_out = gain_out;
  a.alpha_out = alpha_or_null;
  std::vector<ModEntry> tab(n_modules);
  int64_t t0 = 0, items = 0;
  for (int m = 0; m < n_modules; ++m) {
    const int64_t nb = cols[m] / p->C;
    ModEntry& e = tab[m];
    e.W = W[m]; e.W0 = W0[m]; e.d = d[m];
    e.rows = rows[m]; e.cols = cols[m];
    e.tile_off = t0; e.item_off = items; e.pad_ = 0;
    t0 += rows[m] * nb;
    items += (rows[m] + kPeRows - 1) / kPeRows * nb;
  }
  if (items > (int64_t)INT32_MAX) return fail(AWSRC_EINVAL, "too many work items");
  HIPCHK(launch_mod_table(tab.data(), n_modules, mods, s));
  HIPCHK(launch_scored_zero(a.scored, s));  // the pruned screen adds its count
  HIPCHK(launch_gen_basis(p->basis_key, p->C, p->P, p->S, p->gen_version, a.basis, s));
  HIPCHK(launch_pe_screen(a, mods, n_modules, items, a.frag, colsh, s));
  HIPCHK(launch_finalize_pe_modules(a, mods, n_modules, items, s));
  return AWSRC_OK;
}

}  // namespace

extern "C" awsrc_status awsrc_encode_tiles(const awsrc_params* p, const void* W, int32_t w_dtype,
                                           const float* W0, int64_t rows, int64_t cols, const float* d,
                                           int32_t d_mode, uint16_t* seed_out, int8_t* code_out,
                                           uint16_t* scale_out, double* gain_out, float* alpha_or_null,
                                           void* workspace, size_t* ws_bytes, void* stream) {
  const void* Wm[1] = {W};
  const float* W0m[1] = {W0};
  const float* dm[1] = {d};
  const int64_t rm[1] = {rows}, cm[1] = {cols};
  return encode_modules(p, 1, Wm, w_dtype, W0m, dm, d_mode, rm, cm, seed_out, code_out, scale_out, gain_out,
                        alpha_or_null, workspace, ws_bytes, stream);
}

extern "C" awsrc_status awsrc_encode_screen_lists(const awsrc_params* p, int32_t n_modules, const int64_t* rows,
                                                  const int64_t* cols, int32_t d_mode, const void* workspace,
                                                  float* gain_out, uint32_t* seed_out, int32_t* nsplit,
                                                  void* stream) {
  awsrc_status st = check_params(p);
  if (st) return st;
  if (!workspace || !nsplit) return fail(AWSRC_EINVAL, "NULL argument");
  if (d_mode != AWSRC_D_PER_COL && d_mode != AWSRC_D_PER_ELEM) return fail(AWSRC_EINVAL, "bad d_mode %d", d_mode);
  if (n_modules < 1 || !rows || !cols) return fail(AWSRC_EINVAL, "bad module table");
  int64_t T_total = 0;
  for (int m = 0; m < n_modules; ++m) {
    if (rows[m] < 0 || cols[m] < 1 || cols[m] % p->C) return fail(AWSRC_EINVAL, "module %d: bad shape", m);
    T_total += rows[m] * (cols[m] / p->C);
  }
  const char* ws = reinterpret_cast<const char*>(align_up(reinterpret_cast<uintptr_t>(workspace), 256));
  hipStream_t s = (hipStream_t)stream;
  if (pe_batched_supported(p->C, p->P, d_mode, p->gen_version)) {
    // work-item-major lists, permuted into tile order on the device
    const int64_t items = pe_items(p, n_modules, rows, cols);
    const PeLayout l = pe_layout(p, n_modules, items);
    const ModEntry* mods = reinterpret_cast<const ModEntry*>(ws + 256 + l.basis + l.frag + l.colsh);
    const float* tg = reinterpret_cast<const float*>(ws + 256 + l.basis + l.frag + l.colsh + l.mods);
    const uint32_t* ts = reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(tg) + l.tg);
    *nsplit = 1;
    if (!gain_out && !seed_out) return AWSRC_OK;
    if (!gain_out || !seed_out) return fail(AWSRC_EINVAL, "NULL output");
    HIPCHK(launch_pe_lists_tile_order(tg, ts, mods, n_modules, items, gain_out, seed_out, s));
    return AWSRC_OK;
  }
  if (n_modules != 1) return fail(AWSRC_EINVAL, "lists of several modules on the per-module path are not kept");
  const int ns = screen_nsplit(p->C, p->P, p->S, rows[0], cols[0], d_mode, p->gen_version);
  if (screen_fuses_rescore(p->C, p->P, d_mode, p->gen_version, ns))
    return fail(AWSRC_EINVAL, "this screen runs the re-score itself and keeps no lists");
  const int64_t nb = cols[0] / p->C;
  const int PB = factor_pb(p->C, p->P);
  size_t off = 256 + align_up(basis_bytes(p->S, p->P), 256);
  if (d_mode == AWSRC_D_PER_COL) off += align_up((size_t)nb * p->S * colfac_stride(PB) * 4, 256) + align_up((size_t)nb * p->C * 8, 256);
  if (screen_mfma_supported(p->C, p->P, d_mode, p->gen_version)) off += align_up(mfma_frag_bytes(p->C, p->S), 256);
  const float* tg = reinterpret_cast<const float*>(ws + off);
  const uint32_t* ts = reinterpret_cast<const uint32_t*>(ws + off + align_up((size_t)T_total * ns * kTop * 4, 256));
  *nsplit = ns;
  if (!gain_out && !seed_out) return AWSRC_OK;
  if (!gain_out || !seed_out) return fail(AWSRC_EINVAL, "NULL output");
  const size_t n = (size_t)T_total * ns * kTop;
  HIPCHK(hipMemcpyAsync(gain_out, tg, n * 4, hipMemcpyDeviceToDevice, s));
  HIPCHK(hipMemcpyAsync(seed_out, ts, n * 4, hipMemcpyDeviceToDevice, s));
  return AWSRC_OK;
}

extern "C" awsrc_status awsrc_encode_modules(const awsrc_params* p, int32_t n_modules, const void* const* W,
                                             int32_t w_dtype, const float* const* W0, const float* const* d,
                                             int32_t d_mode, const int64_t* rows, const int64_t* cols,
                                             uint16_t* seed_out, int8_t* code_out, uint16_t* scale_out,
                                             double* gain_out, float* alpha_or_null, void* workspace,
                                             size_t* ws_bytes, void* stream) {
  if (n_modules >= 1 && (!W || !W0 || !d) && workspace) return fail(AWSRC_EINVAL, "NULL module pointer array");
  return encode_modules(p, n_modules, W, w_dtype, W0, d, d_mode, rows, cols, seed_out, code_out, scale_out, gain_out,
                        alpha_or_null, workspace, ws_bytes, stream);
}

// ---------------------------------------------------------------- encode, no allocation
namespace {

// Scratch of awsrc_encode_tiles_noalloc: one copy per GPU, held from the
// library's load until the process ends.  In host code `scratch` only names
// the symbol; its device address on the current GPU comes from
// hipGetSymbolAddress, looked up once per device and kept in g_scratch_ptr.
constexpr size_t kNoallocScratchBytes = size_t(64) << 20;
__device__ __attribute__((aligned(256))) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

awsrc_status device_scratch(void** out) {
  int dev = -1;
  HIPCHK(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(AWSRC_EINVAL, "device %d out of range", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    HIPCHK(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
    if (!ptr) return fail(AWSRC_EDEVICE, "no device address for the scratch array");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return AWSRC_OK;
}

}  // namespace

extern "C" uint64_t awsrc_encode_noalloc_max_bytes(void) { return kNoallocScratchBytes; }

extern "C" awsrc_status awsrc_encode_tiles_noalloc(const awsrc_params* p, const void* W, int32_t w_dtype,
                                                   const float* W0, int64_t rows, int64_t cols, const float* d,
                                                   int32_t d_mode, uint16_t* seed_out, int8_t* code_out,
                                                   uint16_t* scale_out, double* gain_out, float* alpha_or_null,
                                                   void* stream) {
  // the size query validates every argument that does not need the device
  size_t need = 0;
  awsrc_status st = awsrc_encode_tiles(p, W, w_dtype, W0, rows, cols, d, d_mode, seed_out, code_out, scale_out,
                                       gain_out, alpha_or_null, nullptr, &need, stream);
  if (st) return st;
  if (need > kNoallocScratchBytes)
    return fail(AWSRC_ENOSPC, "module needs %zu bytes of scratch, more than the %zu-byte static array", need,
                kNoallocScratchBytes);
  if (rows == 0) return AWSRC_OK;
  void* ws = nullptr;
  st = device_scratch(&ws);
  if (st) return st;
  size_t n = kNoallocScratchBytes;
  return awsrc_encode_tiles(p, W, w_dtype, W0, rows, cols, d, d_mode, seed_out, code_out, scale_out, gain_out,
                            alpha_or_null, ws, &n, stream);
}

extern "C" awsrc_status awsrc_sdq_encode(const uint16_t* scale_f16, int64_t n_groups, int8_t* code,
                                         float* block_mean, float* block_step, void* stream) {
  if (n_groups < 0) return fail(AWSRC_EINVAL, "n_groups < 0");
  if (n_groups == 0) return AWSRC_OK;
  if (!scale_f16 || !code || !block_mean || !block_step) return fail(AWSRC_EINVAL, "NULL buffer");
  HIPCHK(launch_sdq_encode(scale_f16, n_groups, code, block_mean, block_step, (hipStream_t)stream));
  return AWSRC_OK;
}

extern "C" awsrc_status awsrc_backbone_sdq_dequant(const uint8_t* codes, const uint8_t* zero, const int8_t* sdq_code,
                                                  const float* block_mean, const float* block_step, int64_t rows,
                                                  int64_t cols, int32_t group, float* W0, void* stream) {
  if (rows < 0 || cols < 0) return fail(AWSRC_EINVAL, "negative shape");
  if (group != 64 && group != 128 && group != 256) return fail(AWSRC_EINVAL, "group must be 64, 128 or 256");
  if (cols % group) return fail(AWSRC_EINVAL, "cols=%lld is not a multiple of group=%d", (long long)cols, group);
  if (rows == 0 || cols == 0) return AWSRC_OK;
  if (!codes || !zero || !sdq_code || !block_mean || !block_step || !W0) return fail(AWSRC_EINVAL, "NULL buffer");
  if ((reinterpret_cast<uintptr_t>(codes) & 3) || (reinterpret_cast<uintptr_t>(W0) & 15))
    return fail(AWSRC_EINVAL, "codes must be 4-byte and W0 16-byte aligned");
  HIPCHK(launch_sdq_dequant(codes, zero, sdq_code, block_mean, block_step, rows, cols, group, W0, (hipStream_t)stream));
  return AWSRC_OK;
}

extern "C" awsrc_status awsrc_encode_scored(const void* workspace, uint64_t* scored, void* stream) {
  if (!workspace || !scored) return fail(AWSRC_EINVAL, "NULL argument");
  const char* ws = reinterpret_cast<const char*>(align_up(reinterpret_cast<uintptr_t>(workspace), 256));
  hipStream_t s = (hipStream_t)stream;
  uint64_t v = 0;
  HIPCHK(hipMemcpyAsync(&v, ws, 8, hipMemcpyDeviceToHost, s));
  HIPCHK(hipStreamSynchronize(s));
  *scored = v;
  return AWSRC_OK;
}

// ---------------------------------------------------------------- rank + serialize
extern "C" awsrc_status awsrc_rank_prefix(const awsrc_params* p, int32_t n_modules,
                                          const int64_t* module_rows, const int64_t* module_cols,
                                          int32_t mode, double bpw_budget, const uint16_t* seed,
                                          const int8_t* code, const uint16_t* scale, const double* gain,
                                          uint8_t* stream_out, uint64_t stream_cap, uint64_t* stream_len,
                                          int64_t* K_out, int64_t* n_eligible, void* workspace,
                                          size_t* ws_bytes, void* stream) {
  awsrc_status st = check_params(p);
  if (st) return st;
  if (!ws_bytes) return fail(AWSRC_EINVAL, "ws_bytes is NULL");
  if (n_modules < 1 || !module_rows || !module_cols) return fail(AWSRC_EINVAL, "bad module table");
  if (mode != AWSRC_MODE_GLOBAL && mode != AWSRC_MODE_PER_MODULE) return fail(AWSRC_EINVAL, "bad mode %d", mode);
  if (!(bpw_budget >= 0.0) || !isfinite(bpw_budget)) return fail(AWSRC_EINVAL, "bpw_budget must be finite and >= 0");
  std::vector<int64_t> toff(n_modules + 1, 0);
  int64_t N = 0;
  for (int m = 0; m < n_modules; ++m) {
    const int64_t r = module_rows[m], c = module_cols[m];
    if (r < 1 || c < 1 || c % p->C) return fail(AWSRC_EINVAL, "module %d: shape %lldx%lld invalid for C=%d", m, (long long)r, (long long)c, p->C);
    if (r > UINT32_MAX || c > UINT32_MAX) return fail(AWSRC_EINVAL, "module %d too large for the header", m);
    toff[m + 1] = toff[m] + r * (c / p->C);
    N += r * c;
  }
  const int64_t T_total = toff[n_modules];
  if (T_total > (int64_t)UINT32_MAX) return fail(AWSRC_EINVAL, "more than 2^32 tiles");
  const int ib = index_bits(p, (uint64_t)T_total);
  if (ib < 32 && (uint64_t)T_total > (1ull << ib)) return fail(AWSRC_EINVAL, "idx_bits=%d cannot address %lld tiles", ib, (long long)T_total);
  const int sb = ceil_log2_u64((uint64_t)p->S);
  const int scb = scale_field_bits(p->scale_fmt);
  const int64_t L = rec_bytes(ib, p->S, p->P, p->b, scb);
  if (L > 255) return fail(AWSRC_EINVAL, "record too large");
  const int64_t h = kHeaderFixed + 8 * (int64_t)n_modules;

  // per-segment record caps from the byte budget
  std::vector<int64_t> seg_t0, seg_n, seg_cap;
  if (mode == AWSRC_MODE_GLOBAL) {
    const int64_t budget = awsrc_budget_bytes(bpw_budget, N);
    if (budget < h) return fail(AWSRC_ENOSPC, "budget %lld bytes < header %lld bytes", (long long)budget, (long long)h);
    seg_t0.push_back(0); seg_n.push_back(T_total); seg_cap.push_back((budget - h) / L);
  } else {
    for (int m = 0; m < n_modules; ++m) {
      seg_t0.push_back(toff[m]);
      seg_n.push_back(toff[m + 1] - toff[m]);
      seg_cap.push_back(awsrc_budget_bytes(bpw_budget, module_rows[m] * module_cols[m]) / L);
    }
  }
  size_t max_n = 0, max_k = 0;
  for (size_t i = 0; i < seg_n.size(); ++i) {
    const int64_t k = seg_cap[i] < seg_n[i] ? seg_cap[i] : seg_n[i];
    if ((size_t)seg_n[i] > max_n) max_n = (size_t)seg_n[i];
    if ((size_t)k > max_k) max_k = (size_t)k;
  }
  const size_t need = 256 + 256 + rank_ws_bytes(max_n, max_k);
  if (!workspace) { *ws_bytes = need; return AWSRC_OK; }
  if (*ws_bytes < need) return fail(AWSRC_ENOSPC, "workspace %zu < %zu bytes", *ws_bytes, need);
  if (!seed || !code || !scale || !gain || !stream_out || !stream_len || !K_out) return fail(AWSRC_EINVAL, "NULL buffer");
  if (stream_cap < (uint64_t)h) return fail(AWSRC_ENOSPC, "stream capacity below the header size");

  char* ws = reinterpret_cast<char*>(align_up(reinterpret_cast<uintptr_t>(workspace), 256));
  const RankWs rw = carve_rank(ws + 256, max_n, max_k);
  hipStream_t s = (hipStream_t)stream;

  // every segment runs on the device back to back (K is found there); one
  // read of the totals at the end
  HIPCHK(launch_rank_init(rw, s));
  for (size_t i = 0; i < seg_n.size(); ++i) {
    const int64_t cap = seg_cap[i] < seg_n[i] ? seg_cap[i] : seg_n[i];
    HIPCHK(launch_rank_segment(gain, seg_t0[i], seg_n[i], cap, rw, seed, code, scale, p->P, p->b, ib, sb, scb, (int)L,
                               (uint64_t)h, stream_cap, stream_out, s));
  }
  // header: fixed fields, then the module table
  std::vector<uint8_t> hdr;
  hdr.reserve(h);
  hdr.push_back('A'); hdr.push_back('W'); hdr.push_back('S'); hdr.push_back('R');
  put_le(hdr, 1, 2);
  put_le(hdr, (uint64_t)(p->gen_version & 0xF) | ((uint64_t)(p->scale_fmt & 0xF) << 4) |
                  ((mode == AWSRC_MODE_PER_MODULE ? 1ull : 0ull) << 8), 2);
  put_le(hdr, (uint64_t)p->C, 2);
  put_le(hdr, (uint64_t)p->P, 1);
  put_le(hdr, (uint64_t)p->b, 1);
  put_le(hdr, (uint64_t)p->S, 4);
  put_le(hdr, (uint64_t)ib, 1);
  put_le(hdr, (uint64_t)sb, 1);
  put_le(hdr, (uint64_t)scb, 1);
  put_le(hdr, (uint64_t)L, 1);
  put_le(hdr, p->basis_key, 8);
  put_le(hdr, (uint64_t)T_total, 8);
  put_le(hdr, (uint64_t)n_modules, 4);
  for (int m = 0; m < n_modules; ++m) {
    put_le(hdr, (uint64_t)module_rows[m], 4);
    put_le(hdr, (uint64_t)module_cols[m], 4);
  }
  // host buffers of this call (the header and the totals) stay alive until
  // the stream synchronization below
  uint64_t tot[3] = {0, 0, 0};
  HIPCHK(hipMemcpyAsync(stream_out, hdr.data(), hdr.size(), hipMemcpyHostToDevice, s));
  HIPCHK(hipMemcpyAsync(tot, rank_totals(rw), 3 * sizeof(uint64_t), hipMemcpyDeviceToHost, s));
  HIPCHK(hipStreamSynchronize(s));
  const int64_t K_total = (int64_t)tot[0];
  if (tot[2]) return fail(AWSRC_ENOSPC, "stream capacity %llu < %lld bytes", (unsigned long long)stream_cap, (long long)(h + K_total * L));
  *stream_len = (uint64_t)(h + K_total * L);
  *K_out = K_total;
  if (n_eligible) *n_eligible = (int64_t)tot[1];
  return AWSRC_OK;
}

// ---------------------------------------------------------------- decode
namespace {

// Workspace: basis tables | tile bitmap with prefix counts | error counter | module tables
// (tile offsets [n+1], cols [n] and W0 pointers [n], contiguous so that one
// host-to-device copy fills them) | decoded records [K] x 32 B | for the bf16
// reconstruction: the records in tile order [K + 1] x 32 B, the prefix-count
// scan scratch, backbone and target pointer tables [3n + 8n].
struct DecodeLayout {
  size_t basis, bitmap, err, tables, dec, dec_t, bsum, bbtab, total;
};

DecodeLayout decode_layout(int S, int P, uint64_t T_total, uint32_t nmod, int64_t K) {
  DecodeLayout l;
  l.basis = align_up(basis_bytes(S, P), 256);
  l.bitmap = align_up((size_t)((T_total + 31) / 32) * 8, 256);
  l.err = 256;
  l.tables = align_up((size_t)(3 * nmod + 1) * 8, 256);
  l.dec = align_up((size_t)K * 32, 256);
  l.dec_t = align_up((size_t)(K + 1) * 32, 256);  // entry 0 is readable even when K = 0
  const size_t nwords = (size_t)((T_total + 31) / 32);
  l.bsum = align_up(((nwords + 4095) / 4096) * 4, 256);
  l.bbtab = align_up((size_t)kBbRows * nmod * 8, 256);
  l.total = 256 + l.basis + l.bitmap + l.err + l.tables + l.dec + l.dec_t + l.bsum + l.bbtab;
  return l;
}

DecodeArgs decode_args(const awsrc_decode_plan* pl) {
  const DecodeLayout l = decode_layout(pl->S, pl->P, pl->T_total, (uint32_t)pl->n_modules, pl->K);
  char* ws = reinterpret_cast<char*>(align_up(reinterpret_cast<uintptr_t>(pl->workspace), 256));
  DecodeArgs a{};
  a.recs = pl->records;
  a.K = pl->K;
  a.C = pl->C; a.P = pl->P; a.b = pl->b; a.S = pl->S;
  a.idx_bits = pl->idx_bits; a.seed_bits = pl->seed_bits; a.L_rec = pl->L_rec;
  a.T_total = pl->T_total;
  a.n_modules = pl->n_modules;
  a.w0_dtype = pl->w0_dtype;
  a.scale_fmt = pl->scale_fmt;
  a.basis = carve_basis(ws, pl->S, pl->P);
  ws += l.basis;
  a.bitmap = reinterpret_cast<uint32_t*>(ws); ws += l.bitmap;
  a.errors = reinterpret_cast<unsigned long long*>(ws); ws += l.err;
  const uint32_t n = (uint32_t)pl->n_modules;
  a.mod_tile_off = reinterpret_cast<const uint64_t*>(ws);
  a.mod_cols = reinterpret_cast<const int64_t*>(ws + 8 * (size_t)(n + 1));
  a.mod_ptr = reinterpret_cast<void* const*>(ws + 8 * (size_t)(2 * n + 1));
  ws += l.tables;
  a.dec = reinterpret_cast<uint4*>(ws);
  ws += l.dec;
  a.dec_t = reinterpret_cast<uint4*>(ws); ws += l.dec_t;
  a.bsum = reinterpret_cast<uint32_t*>(ws);
  return a;
}

}  // namespace

extern "C" awsrc_status awsrc_decode_prepare(const uint8_t* stream_bytes, uint64_t stream_len, int32_t n_modules,
                                             void* const* W0_ptrs, const int64_t* rows, const int64_t* cols,
                                             int32_t w0_dtype, awsrc_decode_plan* plan, void* workspace,
                                             size_t* ws_bytes, void* stream) {
  if (!ws_bytes) return fail(AWSRC_EINVAL, "ws_bytes is NULL");
  if (!stream_bytes) return fail(AWSRC_EINVAL, "stream is NULL");
  if (reinterpret_cast<uintptr_t>(stream_bytes) & 7) return fail(AWSRC_EINVAL, "stream must be 8-byte aligned");
  if (n_modules < 1 || !rows || !cols) return fail(AWSRC_EINVAL, "bad module table");
  if (w0_dtype != AWSRC_DTYPE_F32 && w0_dtype != AWSRC_DTYPE_BF16) return fail(AWSRC_EINVAL, "bad w0_dtype %d", w0_dtype);
  const uint64_t h_caller = kHeaderFixed + 8ull * (uint64_t)n_modules;
  if (stream_len < h_caller) return fail(AWSRC_ECORRUPT, "stream shorter than a header for %d modules", n_modules);
  hipStream_t s = (hipStream_t)stream;
  // host copies of this call (header, module tables, error count) use
  // buffers that live until the stream is synchronized
  std::vector<uint8_t> hbuf(h_caller);
  HIPCHK(hipMemcpyAsync(hbuf.data(), stream_bytes, h_caller, hipMemcpyDeviceToHost, s));
  HIPCHK(hipStreamSynchronize(s));
  const uint8_t* fx = hbuf.data();
  if (memcmp(fx, "AWSR", 4) != 0) return fail(AWSRC_ECORRUPT, "bad magic");
  if (get_le(fx + 4, 2) != 1) return fail(AWSRC_ECORRUPT, "unsupported stream version");
  const uint32_t flags = (uint32_t)get_le(fx + 6, 2);
  const int C = (int)get_le(fx + 8, 2), P = fx[10], b = fx[11];
  const int64_t S = (int64_t)get_le(fx + 12, 4);
  const int ib = fx[16], sb = fx[17], scb = fx[18], L = fx[19];
  const uint64_t key = get_le(fx + 20, 8);
  const uint64_t T_total = get_le(fx + 28, 8);
  const uint32_t nmod = (uint32_t)get_le(fx + 36, 4);
  const int sfmt = (int)((flags >> 4) & 0xF);
  const int gen = (int)(flags & 0xF);
  if ((gen != 1 && gen != 2) || (sfmt != AWSRC_SCALE_FP16 && sfmt != AWSRC_SCALE_POW2) || (flags & ~0x1FFu))
    return fail(AWSRC_ECORRUPT, "bad flags 0x%x", flags);
  if (!pow2_c(C) || P < 1 || P > kMaxP || P > C || b < 2 || b > 8 || S < 2 || S > 65536)
    return fail(AWSRC_ECORRUPT, "bad codec parameters in header");
  if (sb != ceil_log2_u64((uint64_t)S) || scb != scale_field_bits(sfmt) || ib > 32 || (ib == 0 && T_total > 1))
    return fail(AWSRC_ECORRUPT, "bad field widths in header");
  if (L != rec_bytes(ib, (int)S, P, b, scb)) return fail(AWSRC_ECORRUPT, "record size %d inconsistent with header", L);
  if ((int32_t)nmod != n_modules) return fail(AWSRC_ECORRUPT, "header has %u modules, caller %d", nmod, n_modules);
  const uint64_t h = kHeaderFixed + 8ull * nmod;
  if ((stream_len - h) % (uint64_t)L) return fail(AWSRC_ECORRUPT, "stream does not end on a record boundary");
  const uint8_t* mt = fx + kHeaderFixed;
  // host copy of the module tables: tile offsets [n+1] | cols [n] | W0 pointers [n]
  std::vector<uint64_t> tabs(3 * (size_t)nmod + 1, 0);
  uint64_t* toff = tabs.data();
  int64_t* mcols = reinterpret_cast<int64_t*>(tabs.data() + nmod + 1);
  for (uint32_t m = 0; m < nmod; ++m) {
    const int64_t r = (int64_t)get_le(&mt[8 * m], 4), c = (int64_t)get_le(&mt[8 * m + 4], 4);
    if (r != rows[m] || c != cols[m]) return fail(AWSRC_ECORRUPT, "module %u shape %lldx%lld differs from caller's", m, (long long)r, (long long)c);
    if (c % C) return fail(AWSRC_ECORRUPT, "module %u cols not a multiple of C", m);
    toff[m + 1] = toff[m] + (uint64_t)r * (uint64_t)(c / C);
    mcols[m] = c;
  }
  if (toff[nmod] != T_total) return fail(AWSRC_ECORRUPT, "T_total inconsistent with the module table");
  if (ib < 32 && T_total > (1ull << ib)) return fail(AWSRC_ECORRUPT, "index field too narrow");
  const int64_t K = (int64_t)((stream_len - h) / (uint64_t)L);
  const DecodeLayout lay = decode_layout((int)S, P, T_total, nmod, K);
  if (!workspace) { *ws_bytes = lay.total; return AWSRC_OK; }
  if (*ws_bytes < lay.total) return fail(AWSRC_ENOSPC, "workspace %zu < %zu bytes", *ws_bytes, lay.total);
  if (!plan) return fail(AWSRC_EINVAL, "plan is NULL");
  if (!W0_ptrs) return fail(AWSRC_EINVAL, "W0_ptrs is NULL");
  const uintptr_t w0_align = 16;
  for (int m = 0; m < n_modules; ++m) {
    if (!W0_ptrs[m]) return fail(AWSRC_EINVAL, "W0 pointer %d is NULL", m);
    if (reinterpret_cast<uintptr_t>(W0_ptrs[m]) % w0_align)
      return fail(AWSRC_EINVAL, "W0 pointer %d must be 16-byte aligned", m);
  }

  awsrc_decode_plan pl{};
  pl.C = C; pl.P = P; pl.b = b; pl.S = (int32_t)S;
  pl.idx_bits = ib; pl.seed_bits = sb; pl.L_rec = L; pl.n_modules = (int32_t)nmod;
  pl.w0_dtype = w0_dtype;
  pl.scale_fmt = sfmt;
  pl.K = K; pl.T_total = T_total; pl.h = h;
  pl.records = stream_bytes + h;
  pl.workspace = workspace;
  const DecodeArgs a = decode_args(&pl);
  memcpy(tabs.data() + 2 * (size_t)nmod + 1, W0_ptrs, nmod * sizeof(void*));
  HIPCHK(hipMemcpyAsync(const_cast<uint64_t*>(a.mod_tile_off), tabs.data(), tabs.size() * 8, hipMemcpyHostToDevice, s));
  HIPCHK(launch_gen_basis(key, C, P, (int)S, gen, a.basis, s));
  HIPCHK(launch_decode_validate(a, s));
  unsigned long long nerr = 0;
  HIPCHK(hipMemcpyAsync(&nerr, a.errors, 8, hipMemcpyDeviceToHost, s));
  HIPCHK(hipStreamSynchronize(s));
  if (nerr) return fail(AWSRC_ECORRUPT, "%llu invalid or duplicate records", nerr);
  *plan = pl;
  return AWSRC_OK;
}

extern "C" awsrc_status awsrc_decode_apply(const awsrc_decode_plan* plan, void* stream) {
  if (!plan || !plan->workspace) return fail(AWSRC_EINVAL, "plan is NULL or not prepared");
  if (plan->K == 0) return AWSRC_OK;
  HIPCHK(launch_decode_apply(decode_args(plan), (hipStream_t)stream));
  return AWSRC_OK;
}

namespace {

// The dense reconstruction of awsrc_reconstruct_bf16 (n_out == 0, the plan's
// targets) and awsrc_reconstruct_bf16_prefixes (n_out targets of nested
// prefixes).
// scale: fp16 scales, or (sdq_mean and sdq_step not NULL) SDQ scale codes
awsrc_status reconstruct(const awsrc_decode_plan* plan, int32_t n_out, const int64_t* K_out, void* const* out_ptrs,
                         int32_t group, const uint8_t* const* codes, const void* const* scale,
                         const float* const* sdq_mean, const float* const* sdq_step, const uint8_t* const* zero,
                         void* stream) {
  const bool sdq = sdq_mean || sdq_step;
  if (sdq && !(sdq_mean && sdq_step)) return fail(AWSRC_EINVAL, "SDQ block mean and step arrays: both or neither");
  if (!plan || !plan->workspace) return fail(AWSRC_EINVAL, "plan is NULL or not prepared");
  if (n_out == 0 && plan->w0_dtype != AWSRC_DTYPE_BF16) return fail(AWSRC_EINVAL, "the plan's targets must be bf16");
  if (group != 64 && group != 128 && group != 256) return fail(AWSRC_EINVAL, "group=%d: must be 64, 128 or 256", group);
  if (plan->C < 16) return fail(AWSRC_EINVAL, "C=%d: the reconstruction needs C >= 16", plan->C);
  if (!codes || !scale || !zero) return fail(AWSRC_EINVAL, "backbone pointer arrays are NULL");
  const uint32_t n = (uint32_t)plan->n_modules;
  uint32_t kout[kMaxPrefixOutputs] = {};
  for (int o = 0; o < n_out; ++o) {
    if (K_out[o] < 0 || K_out[o] > plan->K)
      return fail(AWSRC_EINVAL, "prefix %d: K=%lld outside 0..%lld", o, (long long)K_out[o], (long long)plan->K);
    kout[o] = (uint32_t)K_out[o];
  }
  const DecodeArgs a = decode_args(plan);
  std::vector<uint64_t> tabs((size_t)kBbRows * n, 0);
  for (uint32_t m = 0; m < n; ++m) {
    if (!codes[m] || !scale[m] || !zero[m]) return fail(AWSRC_EINVAL, "backbone pointer of module %u is NULL", m);
    if (reinterpret_cast<uintptr_t>(codes[m]) & 7) return fail(AWSRC_EINVAL, "codes of module %u must be 8-byte aligned", m);
    if (!sdq && (reinterpret_cast<uintptr_t>(scale[m]) & 1))
      return fail(AWSRC_EINVAL, "scale of module %u must be 2-byte aligned", m);
    tabs[m] = reinterpret_cast<uint64_t>(codes[m]);
    tabs[n + m] = reinterpret_cast<uint64_t>(scale[m]);
    tabs[2 * n + m] = reinterpret_cast<uint64_t>(zero[m]);
    if (sdq) {
      if (!sdq_mean[m] || !sdq_step[m]) return fail(AWSRC_EINVAL, "SDQ block table of module %u is NULL", m);
      if ((reinterpret_cast<uintptr_t>(sdq_mean[m]) | reinterpret_cast<uintptr_t>(sdq_step[m])) & 3)
        return fail(AWSRC_EINVAL, "SDQ block tables of module %u must be 4-byte aligned", m);
      tabs[(size_t)kBbRowSdqMean * n + m] = reinterpret_cast<uint64_t>(sdq_mean[m]);
      tabs[(size_t)kBbRowSdqStep * n + m] = reinterpret_cast<uint64_t>(sdq_step[m]);
    }
    for (int o = 0; o < n_out; ++o) {
      const void* q = out_ptrs[(size_t)o * n + m];
      if (!q) return fail(AWSRC_EINVAL, "target %d of module %u is NULL", o, m);
      if (reinterpret_cast<uintptr_t>(q) & 15) return fail(AWSRC_EINVAL, "target %d of module %u must be 16-byte aligned", o, m);
      tabs[(3 + (size_t)o) * n + m] = reinterpret_cast<uint64_t>(q);
    }
  }
  // stage the backbone pointers and read back the module tables (tile
  // offsets [n+1] then cols [n]); the one synchronization covers both copies
  const DecodeLayout l = decode_layout(plan->S, plan->P, plan->T_total, n, plan->K);
  char* ws = reinterpret_cast<char*>(align_up(reinterpret_cast<uintptr_t>(plan->workspace), 256));
  uint64_t* bbt = reinterpret_cast<uint64_t*>(ws + l.total - 256 - l.bbtab);
  hipStream_t s = (hipStream_t)stream;
  std::vector<uint64_t> mt(2 * (size_t)n + 1, 0);
  HIPCHK(hipMemcpyAsync(bbt, tabs.data(), tabs.size() * 8, hipMemcpyHostToDevice, s));
  HIPCHK(hipMemcpyAsync(mt.data(), a.mod_tile_off, mt.size() * 8, hipMemcpyDeviceToHost, s));
  HIPCHK(hipStreamSynchronize(s));
  for (uint32_t m = 0; m < n; ++m) {
    const int64_t c = (int64_t)mt[n + 1 + m];
    if (c % group) return fail(AWSRC_EINVAL, "module %u: cols %lld not a multiple of group %d", m, (long long)c, group);
    // the kernel indexes units of 16 weights within a module with 32 bits
    if ((mt[m + 1] - mt[m]) * (uint64_t)(plan->C / 16) >= (1ull << 32))
      return fail(AWSRC_EINVAL, "module %u: more than 2^36 weights", m);
  }
  BackboneTabs bb;
  bb.ptr = bbt;
  bb.gshift = group == 64 ? 6 : group == 128 ? 7 : 8;
  bb.sdq = sdq ? 1 : 0;
  HIPCHK(launch_reconstruct_bf16(a, bb, mt.data(), n_out, kout, s));
  return AWSRC_OK;
}

}  // namespace

extern "C" awsrc_status awsrc_reconstruct_bf16(const awsrc_decode_plan* plan, int32_t group,
                                               const uint8_t* const* codes, const uint16_t* const* scale_f16,
                                               const uint8_t* const* zero, void* stream) {
  return reconstruct(plan, 0, nullptr, nullptr, group, codes, reinterpret_cast<const void* const*>(scale_f16), nullptr,
                     nullptr, zero, stream);
}

extern "C" awsrc_status awsrc_reconstruct_bf16_prefixes(const awsrc_decode_plan* plan, int32_t n_out,
                                                        const int64_t* K_out, void* const* out_ptrs, int32_t group,
                                                        const uint8_t* const* codes, const uint16_t* const* scale_f16,
                                                        const uint8_t* const* zero, void* stream) {
  if (n_out < 1 || n_out > kMaxPrefixOutputs) return fail(AWSRC_EINVAL, "n_out=%d: must be 1..%d", n_out, kMaxPrefixOutputs);
  if (!K_out || !out_ptrs) return fail(AWSRC_EINVAL, "K_out or out_ptrs is NULL");
  return reconstruct(plan, n_out, K_out, out_ptrs, group, codes, reinterpret_cast<const void* const*>(scale_f16),
                     nullptr, nullptr, zero, stream);
}

extern "C" awsrc_status awsrc_reconstruct_bf16_sdq(const awsrc_decode_plan* plan, int32_t n_out, const int64_t* K_out,
                                                   void* const* out_ptrs, int32_t group, const uint8_t* const* codes,
                                                   const int8_t* const* sdq_code, const float* const* sdq_mean,
                                                   const float* const* sdq_step, const uint8_t* const* zero,
                                                   void* stream) {
  if (n_out < 0 || n_out > kMaxPrefixOutputs) return fail(AWSRC_EINVAL, "n_out=%d: must be 0..%d", n_out, kMaxPrefixOutputs);
  if (n_out > 0 && (!K_out || !out_ptrs)) return fail(AWSRC_EINVAL, "K_out or out_ptrs is NULL");
  if (!sdq_code || !sdq_mean || !sdq_step) return fail(AWSRC_EINVAL, "SDQ pointer arrays are NULL");
  return reconstruct(plan, n_out, K_out, out_ptrs, group, codes, reinterpret_cast<const void* const*>(sdq_code),
                     sdq_mean, sdq_step, zero, stream);
}

extern "C" awsrc_status awsrc_decode_add(const uint8_t* stream_bytes, uint64_t stream_len, int32_t n_modules,
                                         void* const* W0_ptrs, const int64_t* rows, const int64_t* cols,
                                         int32_t w0_dtype, void* workspace, size_t* ws_bytes, void* stream) {
  awsrc_decode_plan plan{};
  awsrc_status st = awsrc_decode_prepare(stream_bytes, stream_len, n_modules, W0_ptrs, rows, cols, w0_dtype,
                                         &plan, workspace, ws_bytes, stream);
  if (st != AWSRC_OK || !workspace) return st;
  return awsrc_decode_apply(&plan, stream);
}
