// Host side of the C ABI declared in include/blockgtq.h: argument checking,
// the energy score and greedy allocator (host work), the scalar codebook, the
// layout blob builder, and the launch of the HIP kernels.
#include "blockgtq.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "kernels.h"
#include "layout.h"

using namespace bgtq;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return BGTQ_OK;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(BGTQ_EHIP, "%s: %s", what, hipGetErrorString(e));
}

// ---------------------------------------------------------------- fp16 bits
// Round a double to the nearest fp16 (ties to even); finite inputs only.
uint16_t f64_to_f16_bits(double x) {
  uint16_t sign = std::signbit(x) ? 0x8000 : 0;
  double a = std::fabs(x);
  if (a == 0.0) return sign;
  int e;
  std::frexp(a, &e);          // a = m 2^e, m in [0.5, 1)
  int E = e - 1;              // a = 1.f 2^E
  if (E < -14) E = -14;       // subnormal range shares the 2^-24 quantum
  double quantum = std::ldexp(1.0, E - 10);
  double q = std::nearbyint(a / quantum);  // default rounding: to nearest, ties even
  if (q >= 2048.0) {          // mantissa overflowed into the next binade
    q /= 2.0;
    E += 1;
  }
  if (E > 15) return sign | 0x7C00;   // overflow -> inf
  uint32_t mant = static_cast<uint32_t>(q);
  if (mant < 1024) return sign | static_cast<uint16_t>(mant);  // subnormal
  return sign | static_cast<uint16_t>(((E + 15) << 10) | (mant - 1024));
}

double f16_bits_to_f64(uint16_t h) {
  int exp = (h >> 10) & 0x1F, mant = h & 0x3FF;
  double v = exp == 0 ? std::ldexp(static_cast<double>(mant), -24)
                      : std::ldexp(static_cast<double>(mant + 1024), exp - 25);
  return (h & 0x8000) ? -v : v;
}

// --------------------------------------------------- Gaussian Lloyd-Max quantizer
double npdf(double x) { return std::isfinite(x) ? std::exp(-0.5 * x * x) / std::sqrt(2.0 * M_PI) : 0.0; }
// upper tail Q(x) = P(X > x)
double ntail(double x) { return 0.5 * std::erfc(x / std::sqrt(2.0)); }

double prob_between(double lo, double hi) {
  // P(lo <= X < hi) computed from the tail on the side where it is small
  if (lo >= 0) return ntail(lo) - ntail(hi);
  return ntail(-hi) - ntail(-lo);
}

double inv_normal(double p) {
  double lo = -40.0, hi = 40.0;
  for (int it = 0; it < 200; ++it) {
    double mid = 0.5 * (lo + hi);
    if (1.0 - ntail(mid) < p) lo = mid; else hi = mid;
  }
  return 0.5 * (lo + hi);
}

// Centroids of the 2^b-level minimum-MSE quantizer of N(0,1): fixed point of
// c_k = E[X | t_{k-1} <= X < t_k], t_k = (c_k + c_{k+1}) / 2.  Newton steps on
// F(c) = m(c) - c, whose Jacobian is tridiagonal (Thomas algorithm).
std::vector<double> lloyd_max(int b) {
  const int n = 1 << b;
  std::vector<double> c(n), t(n + 1), m(n), lo_d(n), hi_d(n);
  for (int k = 0; k < n; ++k) c[k] = std::sqrt(3.0) * inv_normal((k + 0.5) / n);
  auto eval = [&](const std::vector<double>& cc) {
    t[0] = -INFINITY;
    t[n] = INFINITY;
    for (int k = 1; k < n; ++k) t[k] = 0.5 * (cc[k - 1] + cc[k]);
    for (int k = 0; k < n; ++k) {
      double p = prob_between(t[k], t[k + 1]);
      m[k] = (npdf(t[k]) - npdf(t[k + 1])) / p;
      lo_d[k] = std::isfinite(t[k]) ? npdf(t[k]) * (m[k] - t[k]) / p : 0.0;        // dm_k/dt_k
      hi_d[k] = std::isfinite(t[k + 1]) ? npdf(t[k + 1]) * (t[k + 1] - m[k]) / p : 0.0;  // dm_k/dt_{k+1}
    }
  };
  std::vector<double> a(n), dg(n), up(n), rhs(n);
  for (int it = 0; it < 300; ++it) {
    eval(c);
    // (I - J) step = m - c; J[k][k-1] = lo_d/2, J[k][k] = (lo_d+hi_d)/2, J[k][k+1] = hi_d/2
    for (int k = 0; k < n; ++k) {
      a[k] = -0.5 * lo_d[k];
      dg[k] = 1.0 - 0.5 * (lo_d[k] + hi_d[k]);
      up[k] = -0.5 * hi_d[k];
      rhs[k] = m[k] - c[k];
    }
    for (int k = 1; k < n; ++k) {
      double w = a[k] / dg[k - 1];
      dg[k] -= w * up[k - 1];
      rhs[k] -= w * rhs[k - 1];
    }
    std::vector<double> step(n);
    step[n - 1] = rhs[n - 1] / dg[n - 1];
    for (int k = n - 2; k >= 0; --k) step[k] = (rhs[k] - up[k] * step[k + 1]) / dg[k];
    double lam = 1.0, mx = 0.0;
    std::vector<double> nc(n);
    for (;;) {  // damp until the centroids stay increasing
      bool mono = true;
      for (int k = 0; k < n; ++k) nc[k] = c[k] + lam * step[k];
      for (int k = 1; k < n; ++k) mono = mono && nc[k] > nc[k - 1];
      if (mono || lam < 1e-6) break;
      lam *= 0.5;
    }
    for (int k = 0; k < n; ++k) {
      mx = std::max(mx, std::fabs(nc[k] - c[k]));
      c[k] = nc[k];
    }
    for (int k = 0; k < n / 2; ++k) {  // exact antisymmetry
      double v = 0.5 * (c[n - 1 - k] - c[k]);
      c[k] = -v;
      c[n - 1 - k] = v;
    }
    if (mx < 1e-15) break;
  }
  return c;
}

struct Codebooks {
  uint16_t c16[kCodebookEntries];
  float thr[kThresholdEntries];
  Codebooks() {
    for (int b = 1; b <= 8; ++b) {
      std::vector<double> c = lloyd_max(b);
      const int n = 1 << b;
      for (int k = 0; k < n; ++k) c16[cb_index(b) + k] = f64_to_f16_bits(c[k]);
      for (int k = 0; k + 1 < n; ++k)
        thr[thr_index(b) + k] = static_cast<float>(
            0.5 * (f16_bits_to_f64(c16[cb_index(b) + k]) + f16_bits_to_f64(c16[cb_index(b) + k + 1])));
    }
  }
};

const Codebooks& codebooks() {
  static const Codebooks cb;  // thread-safe one-time init
  return cb;
}

// ------------------------------------------------------------------ configs
int check_cfg(const bgtq_config* c) {
  if (!c) return fail(BGTQ_EINVAL, "config is NULL");
  if (c->head_dim != kHeadDim) return fail(BGTQ_EUNSUPPORTED, "head_dim %d unsupported (only 128)", c->head_dim);
  if (c->n_layers < 1 || c->batch < 1 || c->n_kv_heads < 1)
    return fail(BGTQ_EINVAL, "n_layers, batch and n_kv_heads must be >= 1");
  if (c->group < 1 || c->group > 8) return fail(BGTQ_EUNSUPPORTED, "group %d outside 1..8", c->group);
  if (c->capacity < kKeyTile || c->capacity % kKeyTile != 0)
    return fail(BGTQ_EINVAL, "capacity %d must be a positive multiple of 64", c->capacity);
  if (c->k_budget < kBlocks || c->k_budget > 8 * kBlocks)
    return fail(BGTQ_EBUDGET, "k_budget %d outside [64, 512]", c->k_budget);
  if (c->v_bits < 1 || c->v_bits > 8) return fail(BGTQ_EINVAL, "v_bits %d outside 1..8", c->v_bits);
  if (c->in_dtype != BGTQ_FP32 && c->in_dtype != BGTQ_BF16) return fail(BGTQ_EINVAL, "in_dtype %d", c->in_dtype);
  return BGTQ_OK;
}

int k_words_of(const bgtq_config* c) { return (2 * c->k_budget + 31) / 32; }

Dims dims_of(const bgtq_config* c, int layer) {
  Dims d;
  d.n_layers = c->n_layers;
  d.batch = c->batch;
  d.n_kv = c->n_kv_heads;
  d.group = c->group;
  d.capacity = c->capacity;
  d.k_words = k_words_of(c);
  d.v_bits = c->v_bits;
  d.in_dtype = c->in_dtype;
  d.layer = layer;
  d.n_lc = layer < 0 ? c->n_layers : 1;
  d.max_ctx = c->capacity;
  return d;
}
Dims dims_of(const bgtq_config* c, int layer, int max_ctx) {
  Dims d = dims_of(c, layer);
  d.max_ctx = max_ctx;
  return d;
}

struct SplitPlan {
  int n_splits, split_len;
};

// Default split count.  The decode kernels run one 16-wave workgroup per CU
// (256 CUs), so a launch of U units x n splits takes ceil(U n / 256) rounds,
// each as long as one split: ceil(split length / 1024) 64-row tile
// iterations per wave plus ~2 iterations of set-up and merge.  The plan
// minimises rounds x split time over n; a single round pays 1.15x for the
// spread of per-row costs (the most expensive row decides it), which a second
// round fills in.  Each split covers at least one tile per wave.
SplitPlan plan_splits(const bgtq_config* c, int n_lc, int max_ctx, int requested) {
  SplitPlan p;
  if (max_ctx <= 0) return {1, 64};
  const int max_splits = (max_ctx + kTile - 1) / kTile;
  int n;
  if (requested > 0) {
    n = std::min(requested, max_splits);
  } else {
    const long units = static_cast<long>(c->n_kv_heads) * c->batch * n_lc;
    const int n_hi = std::max(1, std::min(64, (max_ctx + 1023) / 1024));
    double best = 0.0;
    n = 1;
    for (int k = 1; k <= n_hi; ++k) {
      const int len = ((max_ctx + k - 1) / k + 63) / 64 * 64;
      const long rounds = (units * k + 255) / 256;
      double t = static_cast<double>(rounds) * ((len + 1023) / 1024 + 2);
      if (rounds == 1) t *= 1.15;
      if (k == 1 || t < best) {
        best = t;
        n = k;
      }
    }
  }
  p.split_len = ((max_ctx + n - 1) / n + 63) / 64 * 64;
  p.n_splits = (max_ctx + p.split_len - 1) / p.split_len;
  return p;
}

size_t al256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

// The kernels read the cache with 16-byte loads.
bool cache_aligned(const bgtq_cache* c) {
  const auto a = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; };
  return a(c->k_codes) && a(c->k_norms) && a(c->v_codes) && a(c->v_norms);
}

// Workspace: split counters [n_lc][batch][n_kv] int32, then the split
// partials [n_lc][batch][Hq][n_splits][130] fp32.
size_t ws_counter_bytes(const bgtq_config* c, int n_lc) {
  return al256(static_cast<size_t>(n_lc) * c->batch * c->n_kv_heads * 4);
}
size_t ws_bytes_of(const bgtq_config* c, int n_lc, const SplitPlan& p) {
  const size_t hq = static_cast<size_t>(c->n_kv_heads) * c->group;
  const size_t units = static_cast<size_t>(n_lc) * c->batch * hq;
  return ws_counter_bytes(c, n_lc) + al256(units * p.n_splits * 130 * 4);
}

}  // namespace

extern "C" {

const char* blockgtq_last_error(void) { return g_err.c_str(); }

int blockgtq_energy_scores(const float* h_q, const float* h_k, int32_t n_tokens, int32_t group,
                           int32_t head_dim, double* h_scores_out) {
  if (!h_q || !h_k || !h_scores_out) return fail(BGTQ_EINVAL, "NULL pointer");
  if (n_tokens < 1 || group < 1 || head_dim < 2 || head_dim % 2)
    return fail(BGTQ_EINVAL, "bad shape n_tokens=%d group=%d head_dim=%d", n_tokens, group, head_dim);
  const int L = head_dim / 2;
  for (int i = 0; i < L; ++i) {
    double qs = 0.0, ks = 0.0;
    for (int t = 0; t < n_tokens; ++t) {
      for (int g = 0; g < group; ++g) {
        const float* q = h_q + (static_cast<size_t>(t) * group + g) * head_dim;
        qs += static_cast<double>(q[i]) * q[i] + static_cast<double>(q[i + L]) * q[i + L];
      }
      const float* k = h_k + static_cast<size_t>(t) * head_dim;
      ks += static_cast<double>(k[i]) * k[i] + static_cast<double>(k[i + L]) * k[i + L];
    }
    h_scores_out[i] = 0.5 * (qs / (static_cast<double>(n_tokens) * group) + ks / n_tokens);
  }
  return ok();
}

int blockgtq_allocate(const double* h_scores, int32_t n_rows, int32_t n_blocks, int32_t budget,
                      int32_t b_min, int32_t b_max, uint8_t* h_bits_out) {
  if (!h_scores || !h_bits_out) return fail(BGTQ_EINVAL, "NULL pointer");
  if (n_rows < 0 || n_blocks < 1) return fail(BGTQ_EINVAL, "bad shape");
  if (b_min < 1 || b_max > 8 || b_min > b_max) return fail(BGTQ_EINVAL, "bounds must satisfy 1 <= b_min <= b_max <= 8");
  if (budget < n_blocks * b_min || budget > n_blocks * b_max)
    return fail(BGTQ_EBUDGET, "budget %d outside [%d, %d]", budget, n_blocks * b_min, n_blocks * b_max);
  for (long i = 0; i < static_cast<long>(n_rows) * n_blocks; ++i)
    if (!std::isfinite(h_scores[i]) || h_scores[i] < 0.0)
      return fail(BGTQ_EINVAL, "score %ld is negative or not finite", i);
  // J(b) = sum_i s_i 4^-b_i is separable, and raising block i from b to b + 1
  // lowers it by (3/4) s_i 4^-b, a gain that shrinks as b grows (Sec. 3.2;
  // optimality of the greedy rule, App. A.4).  So the optimal schedule takes
  // the B - L b_min largest of the L (b_max - b_min) candidate gains, each
  // candidate (block i, level b) being "the bit that takes i from b to b + 1",
  // and a block's width is b_min plus its number of chosen candidates.  The
  // gain is ordered by s_i 4^-b (exact: a power-of-two scaling), ties by the
  // lower block index, then the lower level (which a block takes first).
  struct Cand {
    double gain;
    int block, level;
  };
  const auto before = [](const Cand& x, const Cand& y) {
    if (x.gain != y.gain) return x.gain > y.gain;
    if (x.block != y.block) return x.block < y.block;
    return x.level < y.level;
  };
  const int extra = budget - n_blocks * b_min;
  std::vector<Cand> cand;
  cand.reserve(static_cast<size_t>(n_blocks) * (b_max - b_min));
  for (int r = 0; r < n_rows; ++r) {
    const double* s = h_scores + static_cast<size_t>(r) * n_blocks;
    uint8_t* bits = h_bits_out + static_cast<size_t>(r) * n_blocks;
    cand.clear();
    for (int i = 0; i < n_blocks; ++i) {
      bits[i] = static_cast<uint8_t>(b_min);
      for (int b = b_min; b < b_max; ++b) cand.push_back({std::ldexp(s[i], -2 * b), i, b});
    }
    if (extra > 0) {
      if (extra < static_cast<int>(cand.size())) std::nth_element(cand.begin(), cand.begin() + extra, cand.end(), before);
      for (int k = 0; k < extra; ++k) ++bits[cand[k].block];
    }
  }
  return ok();
}

int blockgtq_codebook(int32_t b, uint16_t* h_c16_out, float* h_thr_out) {
  if (b < 1 || b > 8) return fail(BGTQ_EINVAL, "b %d outside 1..8", b);
  const Codebooks& cb = codebooks();
  if (h_c16_out) std::memcpy(h_c16_out, cb.c16 + cb_index(b), sizeof(uint16_t) << b);
  if (h_thr_out) std::memcpy(h_thr_out, cb.thr + thr_index(b), sizeof(float) * ((1 << b) - 1));
  return ok();
}

int blockgtq_layout_bytes(const bgtq_config* cfg, size_t* bytes_out) {
  if (int e = check_cfg(cfg)) return e;
  if (!bytes_out) return fail(BGTQ_EINVAL, "NULL pointer");
  *bytes_out = layout_total_bytes(cfg->n_layers * cfg->n_kv_heads);
  return ok();
}

int blockgtq_cache_bytes(const bgtq_config* cfg, size_t* k_codes, size_t* k_norms, size_t* v_codes,
                         size_t* v_norms) {
  if (int e = check_cfg(cfg)) return e;
  const size_t rows = static_cast<size_t>(cfg->n_layers) * cfg->batch * cfg->n_kv_heads;
  const size_t cap = cfg->capacity;
  if (k_codes) *k_codes = rows * cap * k_words_of(cfg) * 4;
  if (k_norms) *k_norms = rows * kMaxGroups * cap * 2;
  if (v_codes) *v_codes = rows * cap * kHeadDim * cfg->v_bits / 8;
  if (v_norms) *v_norms = rows * cap * 2;
  return ok();
}

int blockgtq_workspace_bytes(const bgtq_config* cfg, int32_t n_layers_in_call, int32_t n_splits,
                             int32_t max_ctx, size_t* bytes_out) {
  if (int e = check_cfg(cfg)) return e;
  if (!bytes_out) return fail(BGTQ_EINVAL, "NULL pointer");
  if (n_layers_in_call != 1 && n_layers_in_call != cfg->n_layers)
    return fail(BGTQ_EINVAL, "n_layers_in_call must be 1 or n_layers");
  if (n_splits < 0 || n_splits > 4096) return fail(BGTQ_EINVAL, "n_splits %d outside 0..4096", n_splits);
  if (max_ctx < 0 || max_ctx > cfg->capacity) return fail(BGTQ_ECAPACITY, "max_ctx %d outside [0, capacity]", max_ctx);
  *bytes_out = ws_bytes_of(cfg, n_layers_in_call, plan_splits(cfg, n_layers_in_call, max_ctx, n_splits));
  return ok();
}

int blockgtq_layout_init(const bgtq_config* cfg, const uint8_t* h_k_bits, const float* h_rot_k,
                         const float* h_rot_v, void* d_layout, void* stream) {
  if (int e = check_cfg(cfg)) return e;
  if (!h_k_bits || !h_rot_k || !h_rot_v || !d_layout) return fail(BGTQ_EINVAL, "NULL pointer");
  const int n_rows = cfg->n_layers * cfg->n_kv_heads;
  const size_t total = layout_total_bytes(n_rows);
  std::vector<uint8_t> blob(total, 0);

  Header* H = reinterpret_cast<Header*>(blob.data());
  H->magic = kMagic;
  H->n_rows = n_rows;
  H->n_kv_heads = cfg->n_kv_heads;
  H->k_words = k_words_of(cfg);
  H->v_bits = cfg->v_bits;
  H->off_c16 = kOffC16;
  H->off_thr = kOffThr;
  H->off_rotv = kOffRotV;
  H->off_rotvt = kOffRotVT;
  H->off_rotkt = kOffRotKT;
  H->off_rows = kOffRows;
  H->off_order = layout_order_offset(n_rows);
  H->off_rowrot = layout_rowrot_offset(n_rows);
  H->total_bytes = total;

  const Codebooks& cb = codebooks();
  std::memcpy(blob.data() + kOffC16, cb.c16, sizeof(cb.c16));
  std::memcpy(blob.data() + kOffThr, cb.thr, sizeof(cb.thr));

  float* rotv = reinterpret_cast<float*>(blob.data() + kOffRotV);
  float* rotvt = reinterpret_cast<float*>(blob.data() + kOffRotVT);
  for (int r = 0; r < kHeadDim; ++r)
    for (int q = 0; q < kHeadDim; ++q) {
      const float v = h_rot_v[r * kHeadDim + q];
      if (!std::isfinite(v)) return fail(BGTQ_EINVAL, "rot_v has a non-finite entry");
      rotv[r * kHeadDim + q] = v;
      rotvt[q * kHeadDim + r] = v;
    }
  float* rotkt = reinterpret_cast<float*>(blob.data() + kOffRotKT);
  for (int dd = 2; dd <= kHeadDim; dd += 2) {
    const float* src = h_rot_k + rotk_index(dd);
    float* dst = rotkt + rotk_index(dd);
    for (int r = 0; r < dd; ++r)
      for (int q = 0; q < dd; ++q) {
        const float v = src[r * dd + q];
        if (!std::isfinite(v)) return fail(BGTQ_EINVAL, "rot_k (d=%d) has a non-finite entry", dd);
        dst[q * dd + r] = v;
      }
  }

  RowMeta* rows = reinterpret_cast<RowMeta*>(blob.data() + kOffRows);
  for (int r = 0; r < n_rows; ++r) {
    const uint8_t* bits = h_k_bits + static_cast<size_t>(r) * kBlocks;
    int sum = 0;
    for (int i = 0; i < kBlocks; ++i) {
      if (bits[i] < 1 || bits[i] > 8) return fail(BGTQ_EINVAL, "row %d block %d: width %d outside 1..8", r, i, bits[i]);
      sum += bits[i];
    }
    if (sum != cfg->k_budget) return fail(BGTQ_EBUDGET, "row %d: widths sum to %d, k_budget is %d", r, sum, cfg->k_budget);
    RowMeta& M = rows[r];
    int p = 0, off = 0, g = 0;
    for (int b = 1; b <= 8; ++b) {
      int start = p;
      for (int i = 0; i < kBlocks; ++i) {
        if (bits[i] != b) continue;
        for (int dim : {i, i + kBlocks}) {
          M.dim[p] = static_cast<uint8_t>(dim);
          M.width[p] = static_cast<uint8_t>(b);
          M.bitoff[p] = static_cast<uint16_t>(off);
          M.grp[p] = static_cast<uint8_t>(g);
          off += b;
          ++p;
        }
      }
      if (p > start) {
        M.g_bits[g] = b;
        M.g_dim[g] = p - start;
        M.g_pos[g] = start;
        ++g;
      }
    }
    M.n_groups = g;
    for (int w = 0, slot = 0; w < g; ++w) {
      const uint32_t nst = static_cast<uint32_t>(M.g_dim[w] + 3) / 4;
      // bit 23: the group's width is at most 2 and the row also holds codes of
      // 4 bits or more, so the group's blocks are among the row's
      // lowest-energy ones (the allocator gave them the fewest bits): the
      // decode multiplies only the hi part of the query into them
      const bool hi_only = M.g_bits[w] <= 2 && M.g_bits[g - 1] >= 4;
      M.gm[M.g_bits[w] - 1] = (1u << 31) | static_cast<uint32_t>(M.bitoff[M.g_pos[w]]) | (nst << 10) |
                              (static_cast<uint32_t>(slot) << 16) | (static_cast<uint32_t>(w) << 20) |
                              (hi_only ? (1u << 23) : 0u);
      slot += static_cast<int>((nst + 15) / 16);
    }
    // decode steps: 4 coordinates of one group per step
    int ns = 0;
    for (int gg = 0; gg < g; ++gg) {
      for (int j = 0; j < M.g_dim[gg]; j += 4) {
        const int pos = M.g_pos[gg] + j;
        const int valid = std::min(4, M.g_dim[gg] - j);
        const bool last = j + 4 >= M.g_dim[gg];
        M.step[ns++] = static_cast<uint32_t>(M.bitoff[pos]) | (static_cast<uint32_t>(M.g_bits[gg]) << 10) |
                       (static_cast<uint32_t>(gg) << 14) | (last ? (1u << 17) : 0u) |
                       (static_cast<uint32_t>(pos) << 19) | (static_cast<uint32_t>(valid) << 26);
      }
    }
    M.n_steps = ns;
    for (int w = 0, s2 = 0; w <= kMaxKWords; ++w) {
      while (s2 < ns && static_cast<int>(M.step[s2] & 1023u) < 32 * w) ++s2;
      M.word_step[w] = s2;
    }
    for (int w = 0; w < kMaxKWords; ++w) {
      int first = kHeadDim;
      for (int q = 0; q < kHeadDim; ++q)
        if (M.bitoff[q] + M.width[q] > 32 * w) {
          first = q;
          break;
        }
      M.word_first[w] = first;
    }
  }
  // per-row rotation blocks and the decode dispatch orders
  const float* rotkt_all = reinterpret_cast<const float*>(blob.data() + kOffRotKT);
  std::vector<double> cost(n_rows);
  for (int r = 0; r < n_rows; ++r) {
    const RowMeta& M = rows[r];
    float* dst = reinterpret_cast<float*>(blob.data() + layout_rowrot_offset(n_rows)) +
                 static_cast<size_t>(r) * kRowRotFloats;
    // decode work estimate of one 64-row tile: fixed part, per-group set-up,
    // per-step cost by code width (relative units; only the order matters)
    static const double kStep[9] = {0, 5.5, 3.75, 9.25, 7.75, 20, 20, 20, 20};
    double c = 180.0;
    for (int g = 0; g < M.n_groups; ++g) {
      const int dg = M.g_dim[g];
      std::memcpy(dst, rotkt_all + rotk_index(dg), sizeof(float) * dg * dg);
      dst += dg * dg;
      c += 15.0 + kStep[M.g_bits[g]] * ((dg + 3) / 4);
    }
    cost[r] = c;
  }
  // dense MFMA-order operands of the prefill quantize kernels
  {
    float* mv = reinterpret_cast<float*>(blob.data() + layout_rotv_mfma_offset(n_rows));
    for (int r = 0; r < kHeadDim; ++r)
      for (int c = 0; c < kHeadDim; ++c) mv[mfma_mat_index(r, c)] = h_rot_v[r * kHeadDim + c];
    for (int r = 0; r < n_rows; ++r) {
      const RowMeta& M = rows[r];
      float* mk = reinterpret_cast<float*>(blob.data() + layout_kdense_offset(n_rows)) +
                  static_cast<size_t>(r) * kMfmaMatFloats;
      for (int g = 0; g < M.n_groups; ++g) {
        const int dg = M.g_dim[g], p0 = M.g_pos[g];
        const float* pi = h_rot_k + rotk_index(dg);  // row-major Pi_dg
        for (int j = 0; j < dg; ++j)
          for (int k = 0; k < dg; ++k) mk[mfma_mat_index(p0 + j, M.dim[p0 + k])] = pi[j * dg + k];
      }
    }
  }
  int32_t* order_all = reinterpret_cast<int32_t*>(blob.data() + layout_order_offset(n_rows));
  int32_t* order_layer = order_all + n_rows;
  const auto by_cost = [&](int a, int b) { return cost[a] > cost[b] || (cost[a] == cost[b] && a < b); };
  std::vector<int> idx(n_rows);
  for (int r = 0; r < n_rows; ++r) idx[r] = r;
  std::sort(idx.begin(), idx.end(), by_cost);
  for (int r = 0; r < n_rows; ++r) order_all[r] = idx[r];
  for (int l = 0; l < cfg->n_layers; ++l) {
    std::vector<int> hs(cfg->n_kv_heads);
    for (int h = 0; h < cfg->n_kv_heads; ++h) hs[h] = l * cfg->n_kv_heads + h;
    std::sort(hs.begin(), hs.end(), by_cost);
    for (int h = 0; h < cfg->n_kv_heads; ++h) order_layer[l * cfg->n_kv_heads + h] = hs[h] - l * cfg->n_kv_heads;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(d_layout, blob.data(), total, hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(layout)");
  e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize(layout)");
  return ok();
}

int blockgtq_quantize_append(const bgtq_config* cfg, const void* d_layout, int32_t layer,
                             const void* d_k, const void* d_v, int32_t n_new,
                             const int32_t* d_write_pos, const bgtq_cache* cache, void* stream) {
  if (int e = check_cfg(cfg)) return e;
  if (!d_layout || !d_write_pos || !cache || !cache->k_codes || !cache->k_norms || !cache->v_codes ||
      !cache->v_norms)
    return fail(BGTQ_EINVAL, "NULL pointer");
  if (!cache_aligned(cache)) return fail(BGTQ_EINVAL, "cache buffers must be 16-byte aligned");
  if (layer < -1 || layer >= cfg->n_layers) return fail(BGTQ_EINVAL, "layer %d out of range", layer);
  if (n_new < 0) return fail(BGTQ_EINVAL, "n_new %d < 0", n_new);
  if (n_new > cfg->capacity) return fail(BGTQ_ECAPACITY, "n_new %d > capacity %d", n_new, cfg->capacity);
  if (n_new == 0) return ok();
  if (!d_k || !d_v) return fail(BGTQ_EINVAL, "NULL pointer");
  if (reinterpret_cast<uintptr_t>(d_k) % 16 != 0 || reinterpret_cast<uintptr_t>(d_v) % 16 != 0)
    return fail(BGTQ_EINVAL, "k and v must be 16-byte aligned");
  CachePtrs c{static_cast<uint32_t*>(cache->k_codes), static_cast<uint16_t*>(cache->k_norms),
              static_cast<uint32_t*>(cache->v_codes), static_cast<uint16_t*>(cache->v_norms)};
  hipError_t e = launch_quantize_append(dims_of(cfg, layer), d_layout, d_k, d_v, n_new, d_write_pos, c,
                                        static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "quantize_append launch");
  return ok();
}

static int check_decode_args(const bgtq_config* cfg, int32_t layer, const void* d_q, const int32_t* d_ctx_len,
                             int32_t max_ctx, float* d_out, void* d_ws, size_t ws_bytes, int32_t n_splits,
                             DecodeWs* ws) {
  if (int e = check_cfg(cfg)) return e;
  if (!d_q || !d_ctx_len || !d_out || !d_ws) return fail(BGTQ_EINVAL, "NULL pointer");
  if (reinterpret_cast<uintptr_t>(d_q) % 4 != 0) return fail(BGTQ_EINVAL, "q must be 4-byte aligned");
  if (layer < -1 || layer >= cfg->n_layers) return fail(BGTQ_EINVAL, "layer %d out of range", layer);
  if (max_ctx < 0 || max_ctx > cfg->capacity) return fail(BGTQ_ECAPACITY, "max_ctx %d outside [0, capacity]", max_ctx);
  if (n_splits < 0 || n_splits > 4096) return fail(BGTQ_EINVAL, "n_splits %d outside 0..4096", n_splits);
  const int n_lc = layer < 0 ? cfg->n_layers : 1;
  const SplitPlan p = plan_splits(cfg, n_lc, max_ctx, n_splits);
  const size_t need = ws_bytes_of(cfg, n_lc, p);
  if (ws_bytes < need) return fail(BGTQ_EWORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, need);
  ws->counters = static_cast<int32_t*>(d_ws);
  ws->part = reinterpret_cast<float*>(static_cast<uint8_t*>(d_ws) + ws_counter_bytes(cfg, n_lc));
  ws->n_splits = p.n_splits;
  ws->split_len = p.split_len;
  return BGTQ_OK;
}

int blockgtq_decode_attn(const bgtq_config* cfg, const void* d_layout, int32_t layer, const void* d_q,
                         const int32_t* d_ctx_len, int32_t max_ctx, const bgtq_cache* cache, float* d_out,
                         void* d_workspace, size_t ws_bytes, int32_t n_splits, void* stream) {
  DecodeWs ws;
  if (int e = check_decode_args(cfg, layer, d_q, d_ctx_len, max_ctx, d_out, d_workspace, ws_bytes, n_splits, &ws))
    return e;
  if (!d_layout || !cache || !cache->k_codes || !cache->k_norms || !cache->v_codes || !cache->v_norms)
    return fail(BGTQ_EINVAL, "NULL pointer");
  if (!cache_aligned(cache)) return fail(BGTQ_EINVAL, "cache buffers must be 16-byte aligned");
  CachePtrs c{static_cast<uint32_t*>(cache->k_codes), static_cast<uint16_t*>(cache->k_norms),
              static_cast<uint32_t*>(cache->v_codes), static_cast<uint16_t*>(cache->v_norms)};
  hipError_t e = launch_decode_packed(dims_of(cfg, layer, max_ctx), d_layout, d_q, d_ctx_len, c, d_out, ws,
                                      static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "decode_attn launch");
  return ok();
}

int blockgtq_decode_attn_noalloc(const bgtq_config* cfg, const void* d_layout, int32_t layer, const void* d_q,
                                 const int32_t* d_ctx_len, int32_t max_ctx, const bgtq_cache* cache, float* d_out,
                                 int32_t n_splits, void* stream) {
  if (int e = check_cfg(cfg)) return e;
  if (layer < -1 || layer >= cfg->n_layers) return fail(BGTQ_EINVAL, "layer %d out of range", layer);
  if (max_ctx < 0 || max_ctx > cfg->capacity) return fail(BGTQ_ECAPACITY, "max_ctx %d outside [0, capacity]", max_ctx);
  if (n_splits < 0 || n_splits > 4096) return fail(BGTQ_EINVAL, "n_splits %d outside 0..4096", n_splits);
  const int n_lc = layer < 0 ? cfg->n_layers : 1;
  const size_t need = ws_bytes_of(cfg, n_lc, plan_splits(cfg, n_lc, max_ctx, n_splits));
  if (need > BGTQ_NOALLOC_SCRATCH_BYTES)
    return fail(BGTQ_EWORKSPACE, "this call needs %zu bytes of workspace, more than the %u-byte static array",
                need, BGTQ_NOALLOC_SCRATCH_BYTES);
  void* ws_ptr = nullptr;
  hipError_t e = noalloc_scratch(&ws_ptr);
  if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
  DecodeWs ws;
  if (int rc = check_decode_args(cfg, layer, d_q, d_ctx_len, max_ctx, d_out, ws_ptr, BGTQ_NOALLOC_SCRATCH_BYTES,
                                 n_splits, &ws))
    return rc;
  if (!d_layout || !cache || !cache->k_codes || !cache->k_norms || !cache->v_codes || !cache->v_norms)
    return fail(BGTQ_EINVAL, "NULL pointer");
  if (!cache_aligned(cache)) return fail(BGTQ_EINVAL, "cache buffers must be 16-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  e = launch_clear_counters(ws.counters, n_lc * cfg->batch * cfg->n_kv_heads, s);
  if (e != hipSuccess) return hip_fail(e, "clear_counters launch");
  CachePtrs c{static_cast<uint32_t*>(cache->k_codes), static_cast<uint16_t*>(cache->k_norms),
              static_cast<uint32_t*>(cache->v_codes), static_cast<uint16_t*>(cache->v_norms)};
  e = launch_decode_packed(dims_of(cfg, layer, max_ctx), d_layout, d_q, d_ctx_len, c, d_out, ws, s);
  if (e != hipSuccess) return hip_fail(e, "decode_attn_noalloc launch");
  return ok();
}

int blockgtq_decode_attn_fp16(const bgtq_config* cfg, int32_t layer, const void* d_q, const int32_t* d_ctx_len,
                              int32_t max_ctx, const void* d_k16, const void* d_v16, float* d_out,
                              void* d_workspace, size_t ws_bytes, int32_t n_splits, void* stream) {
  DecodeWs ws;
  if (int e = check_decode_args(cfg, layer, d_q, d_ctx_len, max_ctx, d_out, d_workspace, ws_bytes, n_splits, &ws))
    return e;
  if (!d_k16 || !d_v16) return fail(BGTQ_EINVAL, "NULL pointer");
  hipError_t e = launch_decode_fp16(dims_of(cfg, layer, max_ctx), d_q, d_ctx_len, d_k16, d_v16, d_out, ws,
                                    static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "decode_attn_fp16 launch");
  return ok();
}

static int check_window(int32_t n_sink, int32_t n_recent) {
  if (n_sink < 0 || n_sink > kMaxSink) return fail(BGTQ_EINVAL, "n_sink %d outside 0..%d", n_sink, kMaxSink);
  if (n_recent < 0 || n_recent > kMaxRecent)
    return fail(BGTQ_EINVAL, "n_recent %d outside 0..%d", n_recent, kMaxRecent);
  return BGTQ_OK;
}

int blockgtq_window_bytes(const bgtq_config* cfg, int32_t n_sink, int32_t n_recent, size_t* bytes_out) {
  if (int e = check_cfg(cfg)) return e;
  if (!bytes_out) return fail(BGTQ_EINVAL, "NULL pointer");
  if (int e = check_window(n_sink, n_recent)) return e;
  *bytes_out = static_cast<size_t>(cfg->n_layers) * cfg->batch * cfg->n_kv_heads * 2 *
               static_cast<size_t>(n_sink + n_recent) * kHeadDim * 2;
  return ok();
}

int blockgtq_window_append(const bgtq_config* cfg, int32_t layer, const void* d_k, const void* d_v, int32_t n_new,
                           const int32_t* d_write_pos, int32_t n_sink, int32_t n_recent, void* d_window,
                           void* stream) {
  if (int e = check_cfg(cfg)) return e;
  if (int e = check_window(n_sink, n_recent)) return e;
  if (layer < -1 || layer >= cfg->n_layers) return fail(BGTQ_EINVAL, "layer %d out of range", layer);
  if (n_new < 0) return fail(BGTQ_EINVAL, "n_new %d < 0", n_new);
  if (n_new > cfg->capacity) return fail(BGTQ_ECAPACITY, "n_new %d > capacity %d", n_new, cfg->capacity);
  if (n_new == 0 || n_sink + n_recent == 0) return ok();
  if (!d_k || !d_v || !d_write_pos || !d_window) return fail(BGTQ_EINVAL, "NULL pointer");
  hipError_t e = launch_window_append(dims_of(cfg, layer), d_k, d_v, n_new, d_write_pos, n_sink, n_recent,
                                      static_cast<_Float16*>(d_window), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "window_append launch");
  return ok();
}

int blockgtq_protected_workspace_bytes(const bgtq_config* cfg, int32_t n_layers_in_call, int32_t n_splits,
                                       int32_t max_ctx, size_t* bytes_out) {
  size_t base = 0;
  if (int e = blockgtq_workspace_bytes(cfg, n_layers_in_call, n_splits, max_ctx, &base)) return e;
  *bytes_out = base + al256(static_cast<size_t>(n_layers_in_call) * cfg->batch * cfg->n_kv_heads * cfg->group * 130 * 4);
  return ok();
}

int blockgtq_decode_attn_protected(const bgtq_config* cfg, const void* d_layout, int32_t layer, const void* d_q,
                                   const int32_t* d_ctx_len, int32_t max_ctx, const bgtq_cache* cache,
                                   const void* d_window, int32_t n_sink, int32_t n_recent, float* d_out,
                                   void* d_workspace, size_t ws_bytes, int32_t n_splits, void* stream) {
  DecodeWs ws;
  if (int e = check_window(n_sink, n_recent)) return e;
  if (int e = check_decode_args(cfg, layer, d_q, d_ctx_len, max_ctx, d_out, d_workspace, ws_bytes, n_splits, &ws))
    return e;
  if (!d_layout || (!d_window && n_sink + n_recent > 0) || !cache || !cache->k_codes || !cache->k_norms ||
      !cache->v_codes || !cache->v_norms)
    return fail(BGTQ_EINVAL, "NULL pointer");
  if (!cache_aligned(cache)) return fail(BGTQ_EINVAL, "cache buffers must be 16-byte aligned");
  const int n_lc = layer < 0 ? cfg->n_layers : 1;
  size_t need = 0;
  blockgtq_protected_workspace_bytes(cfg, n_lc, n_splits, max_ctx, &need);
  if (ws_bytes < need) return fail(BGTQ_EWORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, need);
  float* wpart = reinterpret_cast<float*>(static_cast<uint8_t*>(d_workspace) +
                                          ws_bytes_of(cfg, n_lc, plan_splits(cfg, n_lc, max_ctx, n_splits)));
  ws.wpart = wpart;
  ws.n_sink = n_sink;
  ws.n_recent = n_recent;
  const Dims d = dims_of(cfg, layer, max_ctx);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = launch_window_attn(d, d_q, d_ctx_len, static_cast<const _Float16*>(d_window), n_sink, n_recent,
                                    wpart, s);
  if (e != hipSuccess) return hip_fail(e, "window_attn launch");
  CachePtrs c{static_cast<uint32_t*>(cache->k_codes), static_cast<uint16_t*>(cache->k_norms),
              static_cast<uint32_t*>(cache->v_codes), static_cast<uint16_t*>(cache->v_norms)};
  e = launch_decode_packed(d, d_layout, d_q, d_ctx_len, c, d_out, ws, s);
  if (e != hipSuccess) return hip_fail(e, "decode_attn_protected launch");
  return ok();
}

// Workspace of the pre-RoPE step: the decode workspace, then ctx int32
// [batch], RoPE'd q fp32 [n_layers][batch][Hq][128], k and v fp32
// [n_layers][batch][n_kv][128].
struct StepWs {
  size_t decode, ctx, q, k, v, total;
};
static StepWs step_ws(const bgtq_config* cfg, int32_t max_ctx, int32_t n_splits) {
  StepWs w;
  w.decode = ws_bytes_of(cfg, cfg->n_layers, plan_splits(cfg, cfg->n_layers, max_ctx, n_splits));
  const size_t lb = static_cast<size_t>(cfg->n_layers) * cfg->batch;
  w.ctx = w.decode;
  w.q = w.ctx + al256(4 * static_cast<size_t>(cfg->batch));
  w.k = w.q + al256(lb * cfg->n_kv_heads * cfg->group * kHeadDim * 4);
  w.v = w.k + al256(lb * cfg->n_kv_heads * kHeadDim * 4);
  w.total = w.v + al256(lb * cfg->n_kv_heads * kHeadDim * 4);
  return w;
}

int blockgtq_rope_step_workspace_bytes(const bgtq_config* cfg, int32_t max_ctx, int32_t n_splits,
                                       size_t* bytes_out) {
  if (int e = check_cfg(cfg)) return e;
  if (!bytes_out) return fail(BGTQ_EINVAL, "NULL pointer");
  if (n_splits < 0 || n_splits > 4096) return fail(BGTQ_EINVAL, "n_splits %d outside 0..4096", n_splits);
  if (max_ctx < 0 || max_ctx > cfg->capacity) return fail(BGTQ_ECAPACITY, "max_ctx %d outside [0, capacity]", max_ctx);
  *bytes_out = step_ws(cfg, max_ctx, n_splits).total;
  return ok();
}

int blockgtq_rope_decode_step(const bgtq_config* cfg, const void* d_layout, double rope_base, const void* d_q_pre,
                              const void* d_k_pre, const void* d_v, const int32_t* d_pos, int32_t max_ctx,
                              const bgtq_cache* cache, float* d_out, void* d_workspace, size_t ws_bytes,
                              int32_t n_splits, void* stream) {
  if (int e = check_cfg(cfg)) return e;
  if (!d_layout || !d_q_pre || !d_k_pre || !d_v || !d_pos || !d_out || !d_workspace || !cache || !cache->k_codes ||
      !cache->k_norms || !cache->v_codes || !cache->v_norms)
    return fail(BGTQ_EINVAL, "NULL pointer");
  if (!cache_aligned(cache)) return fail(BGTQ_EINVAL, "cache buffers must be 16-byte aligned");
  if (!(rope_base > 1.0) || !std::isfinite(rope_base)) return fail(BGTQ_EINVAL, "rope_base must be finite and > 1");
  if (n_splits < 0 || n_splits > 4096) return fail(BGTQ_EINVAL, "n_splits %d outside 0..4096", n_splits);
  if (max_ctx < 1 || max_ctx > cfg->capacity) return fail(BGTQ_ECAPACITY, "max_ctx %d outside [1, capacity]", max_ctx);
  const StepWs w = step_ws(cfg, max_ctx, n_splits);
  if (ws_bytes < w.total) return fail(BGTQ_EWORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, w.total);
  uint8_t* base = static_cast<uint8_t*>(d_workspace);
  int32_t* ctx = reinterpret_cast<int32_t*>(base + w.ctx);
  float* qo = reinterpret_cast<float*>(base + w.q);
  float* ko = reinterpret_cast<float*>(base + w.k);
  float* vo = reinterpret_cast<float*>(base + w.v);
  Dims d = dims_of(cfg, -1, max_ctx);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = launch_rope_step(d, rope_base, d_q_pre, d_k_pre, d_v, d_pos, qo, ko, vo, ctx, s);
  if (e != hipSuccess) return hip_fail(e, "rope_step launch");
  d.in_dtype = BGTQ_FP32;  // the append and the decode read the fp32 RoPE'd rows
  CachePtrs c{static_cast<uint32_t*>(cache->k_codes), static_cast<uint16_t*>(cache->k_norms),
              static_cast<uint32_t*>(cache->v_codes), static_cast<uint16_t*>(cache->v_norms)};
  e = launch_quantize_append(d, d_layout, ko, vo, 1, d_pos, c, s);
  if (e != hipSuccess) return hip_fail(e, "rope_step append launch");
  const SplitPlan p = plan_splits(cfg, cfg->n_layers, max_ctx, n_splits);
  DecodeWs ws;
  ws.counters = static_cast<int32_t*>(d_workspace);
  ws.part = reinterpret_cast<float*>(base + ws_counter_bytes(cfg, cfg->n_layers));
  ws.n_splits = p.n_splits;
  ws.split_len = p.split_len;
  e = launch_decode_packed(d, d_layout, qo, ctx, c, d_out, ws, s);
  if (e != hipSuccess) return hip_fail(e, "rope_step decode launch");
  return ok();
}

int blockgtq_prefill_workspace_bytes(const bgtq_config* cfg, int32_t n_q, size_t* bytes_out) {
  if (int e = check_cfg(cfg)) return e;
  if (!bytes_out) return fail(BGTQ_EINVAL, "NULL pointer");
  if (n_q < 0) return fail(BGTQ_EINVAL, "n_q %d < 0", n_q);
  *bytes_out = al256(static_cast<size_t>(cfg->batch) * n_q * cfg->n_kv_heads * cfg->group * kHeadDim * 4);
  return ok();
}

int blockgtq_prefill_attn(const bgtq_config* cfg, const void* d_layout, int32_t layer, const void* d_q,
                          int32_t n_q, const int32_t* d_q_pos0, int32_t max_pos, const bgtq_cache* cache,
                          float* d_out, void* d_workspace, size_t ws_bytes, void* stream) {
  if (int e = check_cfg(cfg)) return e;
  if (layer < 0 || layer >= cfg->n_layers) return fail(BGTQ_EINVAL, "layer %d out of range (one layer per call)", layer);
  if (n_q < 0) return fail(BGTQ_EINVAL, "n_q %d < 0", n_q);
  if (n_q == 0) return ok();
  if (!d_layout || !d_q || !d_q_pos0 || !d_out || !d_workspace || !cache || !cache->k_codes || !cache->k_norms ||
      !cache->v_codes || !cache->v_norms)
    return fail(BGTQ_EINVAL, "NULL pointer");
  if (!cache_aligned(cache)) return fail(BGTQ_EINVAL, "cache buffers must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(d_q) % 4 != 0) return fail(BGTQ_EINVAL, "q must be 4-byte aligned");
  if (max_pos < 0 || max_pos >= cfg->capacity)
    return fail(BGTQ_ECAPACITY, "max_pos %d outside [0, capacity)", max_pos);
  size_t need = 0;
  blockgtq_prefill_workspace_bytes(cfg, n_q, &need);
  if (ws_bytes < need) return fail(BGTQ_EWORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, need);
  CachePtrs c{static_cast<uint32_t*>(cache->k_codes), static_cast<uint16_t*>(cache->k_norms),
              static_cast<uint32_t*>(cache->v_codes), static_cast<uint16_t*>(cache->v_norms)};
  hipError_t e = launch_prefill_attn(dims_of(cfg, layer), d_layout, d_q, n_q, d_q_pos0, max_pos, c,
                                     static_cast<float*>(d_workspace), d_out, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "prefill_attn launch");
  return ok();
}

int blockgtq_read_probe(const void* d_src, size_t bytes, uint32_t* d_sink, void* stream) {
  if (!d_src || !d_sink) return fail(BGTQ_EINVAL, "NULL pointer");
  if (bytes == 0 || bytes % 16 != 0 || reinterpret_cast<uintptr_t>(d_src) % 16 != 0)
    return fail(BGTQ_EINVAL, "bytes must be a positive multiple of 16 and the source 16-byte aligned");
  hipError_t e = launch_read_probe(d_src, bytes, d_sink, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "read_probe launch");
  return ok();
}

}  // extern "C"
