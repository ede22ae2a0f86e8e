// Shard specification: uneven split of a layer's KV groups and FFN columns.
//
// Paper Sec. 4.2.1 assigns tensor-parallel shards to devices greedily by
// performance; Sec. 3.2.2 motivates uneven shards. The rounding rule is the
// largest-remainder rule stated in voltron.h. Host-only code: it includes no
// HIP header, so it also builds and runs with a plain C++ compiler.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <numeric>
#include <vector>

#include "internal.hpp"

namespace vt {

static thread_local char g_err[512];

vt_status fail(vt_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return s;
}

void clear_error() { g_err[0] = 0; }

const char* last_error() { return g_err; }

vt_status check_layer_dims(const vt_layer_dims& d) {
  if (d.hidden <= 0 || d.n_heads <= 0 || d.n_kv_heads <= 0 || d.head_dim <= 0 || d.ffn < 0)
    return fail(VT_ERR_ARG, "layer dims must be positive (hidden %d heads %d kv %d head_dim %d ffn %d)",
                d.hidden, d.n_heads, d.n_kv_heads, d.head_dim, d.ffn);
  if (d.n_heads % d.n_kv_heads)
    return fail(VT_ERR_ARG, "n_heads %d is not a multiple of n_kv_heads %d", d.n_heads, d.n_kv_heads);
  if (d.head_dim != 64 && d.head_dim != 128)
    return fail(VT_ERR_UNSUPPORTED, "head_dim %d: only 64 and 128 are supported", d.head_dim);
  if (d.hidden % 8)
    return fail(VT_ERR_UNSUPPORTED, "hidden %d must be a multiple of 8", d.hidden);
  if (d.hidden > 16384)
    return fail(VT_ERR_UNSUPPORTED, "hidden %d exceeds 16384", d.hidden);
  if (!(d.rms_eps >= 0.0f) || !std::isfinite(d.rms_eps))
    return fail(VT_ERR_ARG, "rms_eps must be finite and >= 0");
  if (!(d.rope_base > 0.0f) || !std::isfinite(d.rope_base))
    return fail(VT_ERR_ARG, "rope_base must be finite and > 0");
  if (d.window < 0) return fail(VT_ERR_ARG, "window %d < 0", d.window);
  return VT_OK;
}

// Largest-remainder split of ``total`` units by ``frac`` (validated by caller).
static std::vector<int64_t> apportion(int64_t total, const double* frac, int n) {
  std::vector<int64_t> base(n);
  std::vector<double> rem(n);
  int64_t assigned = 0;
  for (int i = 0; i < n; ++i) {
    double q = frac[i] * static_cast<double>(total);
    double f = std::floor(q);
    base[i] = static_cast<int64_t>(f);
    rem[i] = q - f;
    assigned += base[i];
  }
  int64_t left = total - assigned;
  std::vector<int> order(n);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) {
    if (rem[a] != rem[b]) return rem[a] > rem[b];
    return a < b;
  });
  for (int64_t k = 0; k < left && k < n; ++k) base[order[k]] += 1;
  return base;
}

static vt_status check_fracs(const double* f, int n, const char* what) {
  // Compensated sum so the 1e-9 test does not depend on summation order.
  double s = 0.0, c = 0.0;
  for (int i = 0; i < n; ++i) {
    if (!std::isfinite(f[i]) || f[i] < 0.0)
      return fail(VT_ERR_ARG, "%s fraction %d is %g; fractions must be finite and >= 0", what, i, f[i]);
    double y = f[i] - c;
    double t = s + y;
    c = (t - s) - y;
    s = t;
  }
  if (std::fabs(s - 1.0) > 1e-9)
    return fail(VT_ERR_ARG, "%s fractions sum to %.17g, not 1", what, s);
  return VT_OK;
}

}  // namespace vt

extern "C" {

vt_status vt_shard_spec_create(const vt_layer_dims* dims, int32_t n_devices, const double* head_frac,
                               const double* col_frac, int32_t device, vt_shard_spec** out) {
  vt::clear_error();
  if (!dims || !head_frac || !col_frac || !out) return vt::fail(VT_ERR_ARG, "null argument");
  if (n_devices < 1 || n_devices > 4096)
    return vt::fail(VT_ERR_ARG, "n_devices %d outside 1..4096", n_devices);
  if (device < 0 || device >= n_devices)
    return vt::fail(VT_ERR_ARG, "device %d outside 0..%d", device, n_devices - 1);
  vt_status st = vt::check_layer_dims(*dims);
  if (st != VT_OK) return st;
  if ((st = vt::check_fracs(head_frac, n_devices, "head")) != VT_OK) return st;
  if ((st = vt::check_fracs(col_frac, n_devices, "column")) != VT_OK) return st;

  const int32_t group = dims->n_heads / dims->n_kv_heads;
  auto kv = vt::apportion(dims->n_kv_heads, head_frac, n_devices);
  auto cols = vt::apportion(dims->ffn, col_frac, n_devices);
  int64_t kv0 = 0, c0 = 0;
  for (int i = 0; i < device; ++i) {
    kv0 += kv[i];
    c0 += cols[i];
  }
  vt_shard_spec* s = new (std::nothrow) vt_shard_spec;
  if (!s) return vt::fail(VT_ERR_ARG, "out of host memory");
  s->dims = *dims;
  s->info.kv_head_begin = static_cast<int32_t>(kv0);
  s->info.n_kv_heads = static_cast<int32_t>(kv[device]);
  s->info.q_head_begin = static_cast<int32_t>(kv0 * group);
  s->info.n_q_heads = static_cast<int32_t>(kv[device] * group);
  s->info.col_begin = static_cast<int32_t>(c0);
  s->info.n_cols = static_cast<int32_t>(cols[device]);
  *out = s;
  return VT_OK;
}

vt_status vt_shard_spec_query(const vt_shard_spec* spec, vt_layer_dims* dims_out,
                              vt_shard_info* info_out) {
  vt::clear_error();
  if (!spec) return vt::fail(VT_ERR_ARG, "null spec");
  if (dims_out) *dims_out = spec->dims;
  if (info_out) *info_out = spec->info;
  return VT_OK;
}

void vt_shard_spec_destroy(vt_shard_spec* spec) { delete spec; }

const char* vt_status_string(vt_status s) {
  switch (s) {
    case VT_OK: return "ok";
    case VT_ERR_ARG: return "invalid argument";
    case VT_ERR_ALIGN: return "misaligned pointer or leading dimension";
    case VT_ERR_KV_FULL: return "KV cache full";
    case VT_ERR_POS: return "position does not match KV cache length";
    case VT_ERR_HIP: return "HIP runtime error";
    case VT_ERR_UNSUPPORTED: return "unsupported shape";
    case VT_ERR_WORKSPACE: return "workspace missing or too small";
  }
  return "unknown status";
}

const char* vt_last_error(void) { return vt::last_error(); }

}  // extern "C"
