// C ABI of the LLA latent-cache library: host-side validation, split-K
// heuristic and kernel dispatch.  Every check runs before any HIP call, so an
// invalid call launches nothing and touches no output.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <limits>
#include <mutex>

#include "../../include/lla.h"
#include "lla_internal.h"

namespace {

constexpr double kLog2e = 1.4426950408889634;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool ptr_ok(const void* p) { return p != nullptr && aligned16(p); }
bool opt_ptr_ok(const void* p) { return p == nullptr || aligned16(p); }
bool dtype_ok(int t) { return t == LLA_F32 || t == LLA_BF16; }
bool head_ok(int d) { return d >= 32 && d <= 256 && d % 32 == 0; }
bool rank_ok(int r) { return r >= 1 && r <= LLA_MAX_RANK; }
bool cap_ok(int n_max) { return n_max >= LLA_PAGE_TOKENS && n_max % LLA_PAGE_TOKENS == 0; }
bool rope_ok(int d_rope) { return d_rope >= 8 && d_rope <= LLA_MAX_ROPE && d_rope % 8 == 0; }
// The attention kernels address one latent region (n_max slots of r features:
// per (b, h) for the per-head cache, per sequence for the LLA-2D cache) with
// 32-bit byte offsets.
bool region_ok(int n_max, int r, int dtype) {
  return (int64_t)n_max * r * (dtype == LLA_F32 ? 4 : 2) < ((int64_t)1 << 31);
}
bool regions_ok(int n_max, int r_k, int r_v, int d_rope, int dtype) {
  return region_ok(n_max, r_k, dtype) && region_ok(n_max, r_v, dtype) && region_ok(n_max, d_rope, dtype);
}

int64_t gcd64(int64_t a, int64_t b) {
  while (b) {
    const int64_t t = a % b;
    a = b;
    b = t;
  }
  return a;
}

bool mul_ok(int64_t a, int64_t b, int64_t* out) {
  if (a != 0 && b > std::numeric_limits<int64_t>::max() / a) return false;
  *out = a * b;
  return true;
}

int max_splits(int n_ctx) {
  const int pages = (n_ctx + LLA_PAGE_TOKENS - 1) / LLA_PAGE_TOKENS;
  return pages < LLA_MAX_SPLITS ? pages : LLA_MAX_SPLITS;
}

size_t workspace_bytes(int B, int H, int r_v, int n_ctx) {
  const size_t units = (size_t)B * H;
  const size_t counters = (units * sizeof(uint32_t) + 255) / 256 * 256;
  return counters + units * (size_t)max_splits(n_ctx) * (size_t)(r_v + 2) * sizeof(float);
}

// Launch shape of the decode scan: wavefronts per workgroup and the number of
// workgroups each (b, h) context is split over.  One workgroup per (b, h)
// streams best as long as that already gives every compute unit 8 resident
// wavefronts (4-wave workgroups when (b, h) units alone reach that, 8-wave
// ones otherwise); only smaller batches split the context (split-K), up to 8
// wavefronts per compute unit, with every wavefront keeping at least one
// 8-page group (bf16: one 4-page group when that fills more of the machine).
// bf16 workgroups with fewer 8-page groups than wavefronts use the 4-page K
// groups.  LLA_DECODE_WAVES / LLA_DECODE_SPLITS / LLA_DECODE_DEEP /
// LLA_DECODE_HALF / LLA_DECODE_SHORT / LLA_DECODE_SHORT_WAVES /
// LLA_DECODE_SHORT_GROUPS override the choice (for tuning sweeps).
struct DecodeShape {
  int waves, splits, deep, half, shortk;
};

int env_int(const char* name) {
  const char* e = std::getenv(name);
  return e ? std::atoi(e) : 0;
}

constexpr int kShortPages = 16;

// The larger of the 8-row key blocks (content and rotary) and the 8-row value
// groups a (b, h) walks per 8-page group.
int row_blocks_of(int r_k, int r_v, int d_rope) {
  return std::max((r_k + 7) / 8 + d_rope / 8, (r_v + 7) / 8);
}

DecodeShape choose_shape(int units, int n_ctx, bool allow_split, bool bf16, int row_blocks) {
  static const int forced_waves = env_int("LLA_DECODE_WAVES");
  static const int forced_splits = env_int("LLA_DECODE_SPLITS");
  static const int forced_deep = env_int("LLA_DECODE_DEEP");
  static const int forced_half = env_int("LLA_DECODE_HALF");
  static const int forced_short = env_int("LLA_DECODE_SHORT");
  static const int forced_short_waves = env_int("LLA_DECODE_SHORT_WAVES");
  static const int forced_short_groups = env_int("LLA_DECODE_SHORT_GROUPS");
  const int pages = (n_ctx + LLA_PAGE_TOKENS - 1) / LLA_PAGE_TOKENS;
  const int groups = (pages + 7) / 8;
  const long target = 8L * lla::device_cu_count();  // resident wavefronts wanted
  // bf16: the software-pipelined variant (two batches of loads in flight per
  // wavefront, at most 2 wavefronts per SIMD) measured as fast or faster on
  // every decode workload; fp32 keeps the 4-per-SIMD variant.
  DecodeShape sh{4, 1, bf16 ? 1 : 0, 0, 0};
  if ((long)units * 4 < target && groups >= 8) sh.waves = 8;
  if (allow_split && (long)units * sh.waves < target) {
    // splits that bring units * waves * splits to the target, each wavefront
    // keeping at least `cap`'s share of pages
    auto fill = [&](int w, long cap) {
      const long s = (target + (long)units * w - 1) / ((long)units * w);
      return s < cap ? s : (cap > 0 ? cap : 1L);
    };
    long s = fill(sh.waves, groups / sh.waves);
    // bf16: when whole 8-page groups per wavefront fill at most half the
    // target, one 4-page group per wavefront (the two-rows-per-load K phase)
    // reaches further: the same workgroup size first, then 4 wavefronts; ties
    // keep the fewer splits (a batch that nearly fills the machine is not
    // split for a few more resident wavefronts)
    long best = (long)units * sh.waves * s;
    if (bf16 && 2 * best <= target) {
      for (const int w : {sh.waves, 4}) {
        const long s4 = fill(w, pages / (4 * w));
        if ((long)units * w * s4 > best) {
          best = (long)units * w * s4;
          sh.waves = w;
          s = s4;
        }
      }
    }
    sh.splits = (int)s;
  }
  if (forced_waves == 4 || forced_waves == 8) sh.waves = forced_waves;
  if (forced_splits > 0 && allow_split) sh.splits = forced_splits;
  if (sh.splits > max_splits(n_ctx)) sh.splits = max_splits(n_ctx);
  if (sh.splits < 1) sh.splits = 1;
  if (forced_deep) sh.deep = forced_deep > 0 ? 1 : 0;
  // short contexts: fewer 8-page groups per workgroup than wavefronts -> K
  // groups of 4 pages with two feature rows per load, so every wavefront streams
  if (bf16 && sh.deep) {
    const int per = (pages + sh.splits - 1) / sh.splits;
    sh.half = (per + 7) / 8 < sh.waves ? 1 : 0;
    if (forced_half) sh.half = forced_half > 0 ? 1 : 0;
  }
  // at most kShortPages pages: the wavefronts split the feature rows of each
  // 8-page group (one workgroup per (b, h), not split)
  if (bf16 && sh.waves == 4 && sh.splits == 1) {
    sh.shortk = pages <= kShortPages ? 1 : 0;
    if (forced_short) sh.shortk = forced_short > 0 ? 1 : 0;
  }
  // the row-split kernel takes 8 wavefronts (each walking half as many rows)
  // when its workgroups all fit at one per compute unit (8 wavefronts each
  // fill a unit at 2 per SIMD) and there are more row blocks than 4
  // wavefronts take in one pass
  auto short_waves = [&](long workgroups) {
    if (forced_short_waves == 4 || forced_short_waves == 8) return forced_short_waves;
    return workgroups <= lla::device_cu_count() && row_blocks > 4 ? 8 : 4;
  };
  if (sh.shortk && !forced_waves) sh.waves = short_waves(units);
  // Few (b, h) units over a longer context (bf16, split-K allowed): the same
  // row-split kernel over slices of every context, each slice its own
  // workgroup, when that stays within one workgroup per compute unit.  Every
  // wavefront then walks an eighth or a quarter of the rows of each group, so
  // the chain of dependent load batches per call stays short.  (Two workgroups
  // per unit measured slower than the general kernel's shapes.)
  if (bf16 && allow_split && 2L * units * 4 <= target && pages > 8 && forced_short >= 0 &&
      !forced_waves && !forced_splits && !forced_half) {
    // slices of k 8-page groups, the shortest that fits; longer slices only at
    // larger ranks (16-page slices above 16 row blocks, up to 64-page ones
    // above 40: measured faster than the general kernel's shapes there,
    // slower below)
    const int max_groups = forced_short_groups > 0 ? forced_short_groups
                           : row_blocks > 40       ? 8
                           : row_blocks > 16       ? 2
                                                   : 1;
    for (int k = 1; k <= max_groups; ++k) {
      const long s = (pages + 8L * k - 1) / (8L * k);
      if (s > 1 && (long)units * s <= lla::device_cu_count() && s <= max_splits(n_ctx)) {
        sh = DecodeShape{short_waves((long)units * s), (int)s, 1, 0, 1};
        break;
      }
    }
  }
  // Between half and all of the compute units' worth of (b, h) units over up
  // to 128 pages at 16 to 60 row blocks, or up to 32 pages at any rank: the
  // row-split kernel with 8 wavefronts, one workgroup per (b, h) walking all
  // its groups, measured faster than the general kernel's shapes (which split
  // these contexts or give each wavefront whole 8-page groups).
  if (bf16 && !sh.shortk && forced_short >= 0 && !forced_waves && !forced_splits && !forced_half &&
      2L * units > lla::device_cu_count() && units <= lla::device_cu_count() && row_blocks <= 60 &&
      pages <= 128 && (row_blocks >= 16 || pages <= 32))
    sh = DecodeShape{short_waves(units), 1, 1, 0, 1};
  return sh;
}

lla_status hip_status(hipError_t e) { return e == hipSuccess ? LLA_OK : LLA_ERR_HIP; }

}  // namespace

namespace lla {
int device_cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}
}  // namespace lla

extern "C" {

const char* lla_status_string(int status) {
  switch (status) {
    case LLA_OK: return "LLA_OK: success";
    case LLA_ERR_INVALID_ARG: return "LLA_ERR_INVALID_ARG: invalid size, pointer, alignment or value";
    case LLA_ERR_UNSUPPORTED: return "LLA_ERR_UNSUPPORTED: valid arguments not supported by this build";
    case LLA_ERR_WORKSPACE: return "LLA_ERR_WORKSPACE: decode workspace missing or too small";
    case LLA_ERR_HIP: return "LLA_ERR_HIP: the HIP runtime reported an error";
    case LLA_ERR_SCRATCH:
      return "LLA_ERR_SCRATCH: the call needs more than the library's static scratch "
             "(LLA_NOALLOC_SCRATCH_BYTES per device)";
    default: return "unknown lla_status";
  }
}

int lla_abi_version(void) { return LLA_ABI_VERSION; }

lla_status lla_rho(int64_t T, int64_t d_head, int64_t r_k, int64_t r_v, int64_t* num,
                   int64_t* den) {
  if (T <= 0 || d_head <= 0 || r_k <= 0 || r_v <= 0 || !num || !den) return LLA_ERR_INVALID_ARG;
  int64_t n;
  if (!mul_ok(2 * T, d_head, &n) || r_k > std::numeric_limits<int64_t>::max() - r_v)
    return LLA_ERR_INVALID_ARG;
  const int64_t d = r_k + r_v;
  const int64_t g = gcd64(n, d);
  *num = n / g;
  *den = d / g;
  return LLA_OK;
}

lla_status lla_cache_bytes(int64_t layers, int64_t heads, int64_t T, int64_t d_head, int64_t r_k,
                           int64_t r_v, int64_t tokens, int64_t elem_bytes, int latent,
                           int64_t* bytes) {
  if (layers <= 0 || heads <= 0 || T <= 0 || d_head <= 0 || r_k <= 0 || r_v <= 0 || tokens < 0 ||
      elem_bytes <= 0 || !bytes)
    return LLA_ERR_INVALID_ARG;
  int64_t per = 0, v = 0;
  if (latent) {
    if (!mul_ok(r_k + r_v, heads, &per)) return LLA_ERR_INVALID_ARG;
  } else {
    if (!mul_ok(2 * T, heads, &per) || !mul_ok(per, d_head, &per)) return LLA_ERR_INVALID_ARG;
  }
  if (!mul_ok(layers, per, &v) || !mul_ok(v, elem_bytes, &v) || !mul_ok(v, tokens, &v))
    return LLA_ERR_INVALID_ARG;
  *bytes = v;
  return LLA_OK;
}

namespace {
// Slots of M new tokens at positions pos0 .. pos0+M-1: with an eviction budget
// (window > 0) they must fit the cache and land in distinct slots.
bool slots_ok(int M, int n_max, int pos0, int sink, int window) {
  if (pos0 < 0) return false;
  if (window == 0) return sink == 0 && (int64_t)pos0 + M <= n_max;
  if (window < 0 || sink < 0 || (int64_t)sink + window > n_max) return false;
  if ((int64_t)pos0 + M > std::numeric_limits<int>::max()) return false;
  const int64_t first_ring = pos0 > sink ? pos0 : sink;
  const int64_t in_ring = (int64_t)pos0 + M - first_ring;
  return in_ring <= window;
}

lla_status encode_impl(int dtype, int B, int M, int H, int T, int d_head, int r_k, int r_v,
                       const void* x_k, const void* x_v, const void* mu_k, const void* mu_v,
                       const void* wdt_k, const void* wdt_v, void* c_k, void* c_v, int n_max,
                       int pos0, int sink, int window, void* stream) {
  if (!dtype_ok(dtype) || B < 1 || M < 1 || H < 1 || T < 1 || !head_ok(d_head) || !rank_ok(r_k) ||
      !rank_ok(r_v) || !cap_ok(n_max) || !slots_ok(M, n_max, pos0, sink, window))
    return LLA_ERR_INVALID_ARG;
  if ((int64_t)T * d_head > (1 << 20) || (int64_t)B * M > (1 << 30)) return LLA_ERR_INVALID_ARG;
  if (!ptr_ok(x_k) || !ptr_ok(x_v) || !ptr_ok(wdt_k) || !ptr_ok(wdt_v) || !ptr_ok(c_k) ||
      !ptr_ok(c_v) || !opt_ptr_ok(mu_k) || !opt_ptr_ok(mu_v))
    return LLA_ERR_INVALID_ARG;
  lla::EncodeArgs a{};
  a.dtype = dtype;
  a.B = B;
  a.M = M;
  a.H = H;
  a.K = T * d_head;
  a.r[0] = r_k;
  a.r[1] = r_v;
  a.x[0] = x_k;
  a.x[1] = x_v;
  a.mu[0] = mu_k;
  a.mu[1] = mu_v;
  a.wdt[0] = wdt_k;
  a.wdt[1] = wdt_v;
  a.c[0] = c_k;
  a.c[1] = c_v;
  a.n_max = n_max;
  a.pos0 = pos0;
  a.sink = sink;
  a.window = window;
  a.ksplit = 1;
  return hip_status(lla::launch_encode(a, static_cast<hipStream_t>(stream)));
}

lla_status rope_write_impl(int dtype, int B, int M, int H_rope, int d_rope, const void* k_rope,
                           double base, void* r_cache, int n_max, int pos0, int sink, int window,
                           void* stream) {
  if (!dtype_ok(dtype) || B < 1 || M < 1 || H_rope < 1 || H_rope > 65535 || !rope_ok(d_rope) || !cap_ok(n_max) ||
      !slots_ok(M, n_max, pos0, sink, window) || !std::isfinite(base) || !(base > 1.0))
    return LLA_ERR_INVALID_ARG;
  if ((int64_t)B * M * H_rope * d_rope > (1LL << 34) || !ptr_ok(k_rope) || !ptr_ok(r_cache))
    return LLA_ERR_INVALID_ARG;
  lla::RopeArgs a{};
  a.dtype = dtype;
  a.B = B;
  a.G = H_rope;
  a.M = M;
  a.dr = d_rope;
  a.x = k_rope;
  a.pos0 = pos0;
  a.base = base;
  a.y = r_cache;
  a.n_max = n_max;
  a.sink = sink;
  a.window = window;
  return hip_status(lla::launch_rope_write(a, static_cast<hipStream_t>(stream)));
}
}  // namespace

lla_status lla_encode(int dtype, int B, int M, int H, int T, int d_head, int r_k, int r_v,
                      const void* x_k, const void* x_v, const void* mu_k, const void* mu_v,
                      const void* wdt_k, const void* wdt_v, void* c_k, void* c_v, int n_max,
                      int pos0, void* stream) {
  return encode_impl(dtype, B, M, H, T, d_head, r_k, r_v, x_k, x_v, mu_k, mu_v, wdt_k, wdt_v, c_k,
                     c_v, n_max, pos0, 0, 0, stream);
}

lla_status lla_encode_ring(int dtype, int B, int M, int H, int T, int d_head, int r_k, int r_v,
                           const void* x_k, const void* x_v, const void* mu_k, const void* mu_v,
                           const void* wdt_k, const void* wdt_v, void* c_k, void* c_v, int n_max,
                           int pos0, int sink, int window, void* stream) {
  if (window < 1) return LLA_ERR_INVALID_ARG;
  return encode_impl(dtype, B, M, H, T, d_head, r_k, r_v, x_k, x_v, mu_k, mu_v, wdt_k, wdt_v, c_k,
                     c_v, n_max, pos0, sink, window, stream);
}

lla_status lla_decode_workspace_bytes(int B, int H, int r_v, int n_ctx, size_t* bytes) {
  if (B < 1 || H < 1 || !rank_ok(r_v) || n_ctx < 1 || !bytes) return LLA_ERR_INVALID_ARG;
  *bytes = workspace_bytes(B, H, r_v, n_ctx);
  return LLA_OK;
}

lla_status lla_decode_splits(int dtype, int B, int H, int n_ctx, int r_k, int r_v, int d_rope,
                             int with_workspace, int* splits) {
  if (!dtype_ok(dtype) || B < 1 || H < 1 || n_ctx < 1 || !splits || (int64_t)B * H > (1 << 24) ||
      !rank_ok(r_k) || !rank_ok(r_v) || d_rope < 0 || d_rope > LLA_MAX_ROPE)
    return LLA_ERR_INVALID_ARG;
  *splits = choose_shape(B * H, n_ctx, with_workspace != 0, dtype == LLA_BF16,
                         row_blocks_of(r_k, r_v, d_rope)).splits;
  return LLA_OK;
}

namespace {
// ---- static scratch of the allocation-free decode entry point ----
// One array per device (each GPU the library runs on holds its own copy until
// the process ends).  Host code never uses the array's name as an address:
// hipGetSymbolAddress resolves the device address once per device, and that
// pointer is what kernels and fills receive.
constexpr size_t kStaticScratchBytes = LLA_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
struct ScratchSlot {
  std::once_flag once;
  void* ptr = nullptr;
  hipError_t err = hipSuccess;
};
ScratchSlot g_scratch[kMaxDevices];

// Device address of the current device's scratch, resolved on the first call
// on that device (with it current).
lla_status static_scratch_base(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return LLA_ERR_HIP;
  ScratchSlot& slot = g_scratch[dev];
  std::call_once(slot.once, [&slot] {
    slot.err = hipGetSymbolAddress(&slot.ptr, HIP_SYMBOL(scratch));
  });
  if (slot.err != hipSuccess || slot.ptr == nullptr) return LLA_ERR_HIP;
  *out = slot.ptr;
  return LLA_OK;
}

__global__ void zero_u32_kernel(uint32_t* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

lla_status decode_impl(int dtype, int out_dtype, int B, int H, int d_head, int r_k, int r_v,
                       int d_rope, int H_rope, int n_max, int n_ctx, const int32_t* ctx_len,
                       const void* q, const void* q_rope, const void* c_k, const void* c_v,
                       const void* r_cache, const void* u_k, const void* u_v, const void* mu_k,
                       const void* mu_v, float scale, void* out, void* workspace,
                       size_t ws_bytes, void* stream, bool static_scratch = false) {
  if (!dtype_ok(dtype) || !dtype_ok(out_dtype) || B < 1 || H < 1 || !head_ok(d_head) ||
      !rank_ok(r_k) || !rank_ok(r_v) || !cap_ok(n_max) || n_ctx < 1 || n_ctx > n_max ||
      !std::isfinite(scale) || !(scale > 0.f))
    return LLA_ERR_INVALID_ARG;
  if ((int64_t)B * H > (1 << 24)) return LLA_ERR_INVALID_ARG;
  if (!ptr_ok(q) || !ptr_ok(c_k) || !ptr_ok(c_v) || !ptr_ok(u_k) || !ptr_ok(u_v) || !ptr_ok(out) ||
      !opt_ptr_ok(mu_k) || !opt_ptr_ok(mu_v) ||
      (ctx_len && (reinterpret_cast<uintptr_t>(ctx_len) & 3u)))
    return LLA_ERR_INVALID_ARG;
  if (d_rope && (!rope_ok(d_rope) || !(H_rope == 1 || H_rope == H) || !ptr_ok(q_rope) ||
                 !ptr_ok(r_cache) || ((r_k + 7) / 8) * 8 + d_rope > LLA_MAX_RANK))
    return LLA_ERR_INVALID_ARG;
  if (!regions_ok(n_max, r_k, r_v, d_rope, dtype)) return LLA_ERR_UNSUPPORTED;
  if (!static_scratch) {
    if ((workspace == nullptr) != (ws_bytes == 0)) return LLA_ERR_WORKSPACE;
    if (workspace && (!aligned16(workspace) || ws_bytes < workspace_bytes(B, H, r_v, n_ctx)))
      return LLA_ERR_WORKSPACE;
  }
  (void)mu_k;  // q . mu_k is constant over the context: it cancels in the softmax

  lla::DecodeArgs a{};
  a.dtype = dtype;
  a.out_dtype = out_dtype;
  a.B = B;
  a.H = H;
  a.d = d_head;
  a.rk = r_k;
  a.rv = r_v;
  a.n_max = n_max;
  a.n_ctx = n_ctx;
  a.M = 1;
  a.p0 = 0;
  a.causal = 0;
  a.ctx_len = ctx_len;
  a.q = q;
  a.ck = c_k;
  a.cv = c_v;
  a.uk = u_k;
  a.uv = u_v;
  a.muv = mu_v;
  a.qscale = (float)((double)scale * kLog2e);
  a.out = out;
  a.dr = d_rope;
  a.Hr = H_rope;
  a.qr = q_rope;
  a.rc = r_cache;
  const DecodeShape sh = choose_shape(B * H, n_ctx, static_scratch || workspace != nullptr,
                                      dtype == LLA_BF16, row_blocks_of(r_k, r_v, d_rope));
  a.waves = sh.waves;
  a.splits = sh.splits;
  a.deep = sh.deep;
  a.half = sh.half;
  a.shortk = sh.shortk;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  if (static_scratch) {
    // partials of exactly the chosen split count, in the device's static array
    void* base = nullptr;
    const lla_status e = static_scratch_base(&base);
    if (e != LLA_OK) return e;
    if (a.splits > 1) {
      const size_t units = (size_t)B * H;
      const size_t counters = (units * sizeof(uint32_t) + 255) / 256 * 256;
      if (counters + units * a.splits * (size_t)(r_v + 2) * sizeof(float) > kStaticScratchBytes)
        return LLA_ERR_SCRATCH;
      // the arrival counters must start at zero; a fill kernel, not a memset
      // node, so the call can be captured into a graph
      const int n = (int)units;
      hipLaunchKernelGGL(zero_u32_kernel, dim3((n + 255) / 256), dim3(256), 0, st,
                         static_cast<uint32_t*>(base), n);
      if (hipGetLastError() != hipSuccess) return LLA_ERR_HIP;
      a.cnt = static_cast<uint32_t*>(base);
      a.part = reinterpret_cast<float*>(static_cast<char*>(base) + counters);
    }
  } else if (a.splits > 1) {
    const size_t units = (size_t)B * H;
    const size_t counters = (units * sizeof(uint32_t) + 255) / 256 * 256;
    a.cnt = static_cast<uint32_t*>(workspace);
    a.part = reinterpret_cast<float*>(static_cast<char*>(workspace) + counters);
  }
  return hip_status(lla::launch_decode(a, st));
}
}  // namespace

lla_status lla_decode_attn(int dtype, int out_dtype, int B, int H, int d_head, int r_k, int r_v,
                           int n_max, int n_ctx, const int32_t* ctx_len, const void* q,
                           const void* c_k, const void* c_v, const void* u_k, const void* u_v,
                           const void* mu_k, const void* mu_v, float scale, void* out,
                           void* workspace, size_t ws_bytes, void* stream) {
  return decode_impl(dtype, out_dtype, B, H, d_head, r_k, r_v, 0, 1, n_max, n_ctx, ctx_len, q,
                     nullptr, c_k, c_v, nullptr, u_k, u_v, mu_k, mu_v, scale, out, workspace,
                     ws_bytes, stream);
}

lla_status lla_decode_attn_noalloc(int dtype, int out_dtype, int B, int H, int d_head, int r_k,
                                   int r_v, int n_max, int n_ctx, const int32_t* ctx_len,
                                   const void* q, const void* c_k, const void* c_v, const void* u_k,
                                   const void* u_v, const void* mu_k, const void* mu_v, float scale,
                                   void* out, void* stream) {
  return decode_impl(dtype, out_dtype, B, H, d_head, r_k, r_v, 0, 1, n_max, n_ctx, ctx_len, q,
                     nullptr, c_k, c_v, nullptr, u_k, u_v, mu_k, mu_v, scale, out, nullptr, 0,
                     stream, /*static_scratch=*/true);
}

lla_status lla_decode_attn_rope(int dtype, int out_dtype, int B, int H, int d_head, int r_k,
                                int r_v, int d_rope, int H_rope, int n_max, int n_ctx,
                                const int32_t* ctx_len, const void* q, const void* q_rope,
                                const void* c_k, const void* c_v, const void* r_cache,
                                const void* u_k, const void* u_v, const void* mu_k,
                                const void* mu_v, float scale, void* out, void* workspace,
                                size_t ws_bytes, void* stream) {
  if (d_rope < 1) return LLA_ERR_INVALID_ARG;
  return decode_impl(dtype, out_dtype, B, H, d_head, r_k, r_v, d_rope, H_rope, n_max, n_ctx,
                     ctx_len, q, q_rope, c_k, c_v, r_cache, u_k, u_v, mu_k, mu_v, scale, out,
                     workspace, ws_bytes, stream);
}

lla_status lla_decode_attn_fullrope(int dtype, int out_dtype, int B, int H, int d_head, int r_k,
                                    int r_v, int n_max, int n_ctx, const int32_t* ctx_len,
                                    const int32_t* q_pos, const void* q, const void* c_k,
                                    const void* c_v, const void* u_k, const void* u_v,
                                    const void* mu_k, const void* mu_v, double base, float scale,
                                    void* out, void* workspace, size_t ws_bytes, void* stream) {
  if (!dtype_ok(dtype) || !dtype_ok(out_dtype) || B < 1 || H < 1 || !head_ok(d_head) ||
      !rank_ok(r_k) || !rank_ok(r_v) || !cap_ok(n_max) || n_ctx < 1 || n_ctx > n_max ||
      !std::isfinite(scale) || !(scale > 0.f) || !std::isfinite(base) || !(base > 1.0))
    return LLA_ERR_INVALID_ARG;
  if ((int64_t)B * H > (1 << 24)) return LLA_ERR_INVALID_ARG;
  if (!ptr_ok(q) || !ptr_ok(c_k) || !ptr_ok(c_v) || !ptr_ok(u_k) || !ptr_ok(u_v) || !ptr_ok(out) ||
      !opt_ptr_ok(mu_k) || !opt_ptr_ok(mu_v) ||
      (ctx_len && (reinterpret_cast<uintptr_t>(ctx_len) & 3u)) ||
      (q_pos && (reinterpret_cast<uintptr_t>(q_pos) & 3u)))
    return LLA_ERR_INVALID_ARG;
  if (!regions_ok(n_max, r_k, r_v, 0, dtype)) return LLA_ERR_UNSUPPORTED;
  if ((workspace == nullptr) != (ws_bytes == 0)) return LLA_ERR_WORKSPACE;
  if (workspace && (!aligned16(workspace) || ws_bytes < workspace_bytes(B, H, r_v, n_ctx)))
    return LLA_ERR_WORKSPACE;
  lla::FullRopeArgs a{};
  a.dtype = dtype;
  a.out_dtype = out_dtype;
  a.B = B;
  a.H = H;
  a.d = d_head;
  a.rk = r_k;
  a.rv = r_v;
  a.n_max = n_max;
  a.n_ctx = n_ctx;
  a.ctx_len = ctx_len;
  a.q_pos = q_pos;
  a.q = q;
  a.ck = c_k;
  a.cv = c_v;
  a.uk = u_k;
  a.uv = u_v;
  a.muk = mu_k;
  a.muv = mu_v;
  a.base = base;
  a.qscale = (float)((double)scale * kLog2e);
  a.out = out;
  a.splits = 1;
  // Split the context only for the MFMA kernel and only when the (b, h) units
  // alone leave compute units without a resident workgroup; every split keeps
  // at least 4 pages (the prologue forms the rotation constants and loads U_k).
  if (workspace && lla::fullrope_mfma_ok(dtype, d_head, r_k, r_v)) {
    static const int forced = env_int("LLA_FULLROPE_SPLITS");
    const long target = (long)lla::fullrope_occupancy(r_k, r_v) * lla::device_cu_count();
    const long units = (long)B * H;
    long s = units < target ? (target + units - 1) / units : 1;
    const long cap = ((n_ctx + LLA_PAGE_TOKENS - 1) / LLA_PAGE_TOKENS) / 4;
    if (s > cap) s = cap;
    if (forced > 0) s = forced;
    if (s > max_splits(n_ctx)) s = max_splits(n_ctx);
    a.splits = s < 1 ? 1 : (int)s;
  }
  if (a.splits > 1) {
    const size_t units = (size_t)B * H;
    const size_t counters = (units * sizeof(uint32_t) + 255) / 256 * 256;
    a.cnt = static_cast<uint32_t*>(workspace);
    a.part = reinterpret_cast<float*>(static_cast<char*>(workspace) + counters);
  }
  return hip_status(lla::launch_decode_fullrope(a, static_cast<hipStream_t>(stream)));
}

namespace {
// bf16 prefill kernels: the absorbed kernel takes feature tiles up to 96 (one
// of them carries the running max, one the denominator); larger ranks rebuild
// each head's K and V (d_head 128, ranks multiples of 8) into the workspace.
bool prefill_absorbed_ok(int d_head, int r_k, int r_v, int d_rope) {
  return r_k + d_rope <= 95 && r_v <= 95 && d_head <= 128;
}
bool prefill_rebuild_ok(int d_head, int r_k, int r_v, int d_rope) {
  return d_rope == 0 && d_head == 128 && r_k % 8 == 0 && r_v % 8 == 0;
}
size_t prefill_rebuild_bytes(int B, int H, int d_head, int n_keys) {
  const size_t nk = ((size_t)n_keys + LLA_PAGE_TOKENS - 1) / LLA_PAGE_TOKENS * LLA_PAGE_TOKENS;
  return 4 * (size_t)B * H * d_head * nk;  // fp16 K and V
}

lla_status prefill_impl(int dtype, int out_dtype, int B, int H, int M, int d_head, int r_k, int r_v,
                        int d_rope, int H_rope, int n_max, int p0, const void* q,
                        const void* q_rope, const void* c_k, const void* c_v, const void* r_cache,
                        const void* u_k, const void* u_v, const void* mu_k, const void* mu_v,
                        float scale, void* out, void* workspace, size_t ws_bytes, void* stream) {
  if (!dtype_ok(dtype) || !dtype_ok(out_dtype) || B < 1 || H < 1 || M < 1 || !head_ok(d_head) ||
      !rank_ok(r_k) || !rank_ok(r_v) || !cap_ok(n_max) || p0 < 0 || (int64_t)p0 + M > n_max ||
      !std::isfinite(scale) || !(scale > 0.f))
    return LLA_ERR_INVALID_ARG;
  if ((int64_t)B * H * M > (1 << 30)) return LLA_ERR_INVALID_ARG;
  if (!ptr_ok(q) || !ptr_ok(c_k) || !ptr_ok(c_v) || !ptr_ok(u_k) || !ptr_ok(u_v) || !ptr_ok(out) ||
      !opt_ptr_ok(mu_k) || !opt_ptr_ok(mu_v))
    return LLA_ERR_INVALID_ARG;
  if (d_rope && (!rope_ok(d_rope) || !(H_rope == 1 || H_rope == H) || !ptr_ok(q_rope) ||
                 !ptr_ok(r_cache) || ((r_k + 7) / 8) * 8 + d_rope > LLA_MAX_RANK))
    return LLA_ERR_INVALID_ARG;
  if (!regions_ok(n_max, r_k, r_v, d_rope, dtype)) return LLA_ERR_UNSUPPORTED;
  (void)mu_k;  // q . mu_k is constant over the keys of a query: it cancels in the softmax
  const float qscale = (float)((double)scale * kLog2e);
  if ((workspace == nullptr) != (ws_bytes == 0)) return LLA_ERR_WORKSPACE;
  if (dtype == LLA_BF16 && !prefill_absorbed_ok(d_head, r_k, r_v, d_rope)) {
    if (!prefill_rebuild_ok(d_head, r_k, r_v, d_rope) || (M + 255) / 256 > 65535 || (int64_t)B * H > 65535)
      return LLA_ERR_UNSUPPORTED;
    if (!workspace || !aligned16(workspace) || ws_bytes < prefill_rebuild_bytes(B, H, d_head, p0 + M))
      return LLA_ERR_WORKSPACE;
    lla::Prefill2dArgs a{};
    a.out_dtype = out_dtype;
    a.B = B;
    a.H = H;
    a.M = M;
    a.rk = r_k;
    a.rv = r_v;
    a.n_max = n_max;
    a.p0 = p0;
    a.nk = (p0 + M + LLA_PAGE_TOKENS - 1) / LLA_PAGE_TOKENS * LLA_PAGE_TOKENS;
    a.q = q;
    a.ck = c_k;
    a.cv = c_v;
    a.uk = u_k;
    a.uv = u_v;
    a.muv = mu_v;
    a.qscale = qscale;
    a.out = out;
    a.kh = workspace;
    a.vt = static_cast<char*>(workspace) + prefill_rebuild_bytes(B, H, d_head, p0 + M) / 2;
    return hip_status(lla::launch_prefill_rebuild(a, static_cast<hipStream_t>(stream)));
  }
  if (dtype == LLA_BF16) {
    if ((M + 127) / 128 > 65535) return LLA_ERR_UNSUPPORTED;
    lla::PrefillArgs a{};
    a.out_dtype = out_dtype;
    a.B = B;
    a.H = H;
    a.M = M;
    a.d = d_head;
    a.rk = r_k;
    a.rv = r_v;
    a.n_max = n_max;
    a.p0 = p0;
    a.q = q;
    a.ck = c_k;
    a.cv = c_v;
    a.uk = u_k;
    a.uv = u_v;
    a.muv = mu_v;
    a.qscale = qscale;
    a.out = out;
    a.dr = d_rope;
    a.Hr = H_rope;
    a.qr = q_rope;
    a.rc = r_cache;
    return hip_status(lla::launch_prefill_bf16(a, static_cast<hipStream_t>(stream)));
  }
  // fp32: the decode scan, one workgroup per query, query m over [0, p0 + m].
  lla::DecodeArgs a{};
  a.dtype = dtype;
  a.out_dtype = out_dtype;
  a.B = B;
  a.H = H;
  a.d = d_head;
  a.rk = r_k;
  a.rv = r_v;
  a.n_max = n_max;
  a.n_ctx = p0 + M;
  a.M = M;
  a.p0 = p0;
  a.causal = 1;
  a.splits = 1;
  a.waves = 4;
  a.deep = 0;
  a.q = q;
  a.ck = c_k;
  a.cv = c_v;
  a.uk = u_k;
  a.uv = u_v;
  a.muv = mu_v;
  a.qscale = qscale;
  a.out = out;
  a.dr = d_rope;
  a.Hr = H_rope;
  a.qr = q_rope;
  a.rc = r_cache;
  return hip_status(lla::launch_decode(a, static_cast<hipStream_t>(stream)));
}
}  // namespace

lla_status lla_prefill_workspace_bytes(int dtype, int B, int H, int M, int d_head, int r_k, int r_v,
                                      int p0, size_t* bytes) {
  if (!dtype_ok(dtype) || B < 1 || H < 1 || M < 1 || !head_ok(d_head) || !rank_ok(r_k) ||
      !rank_ok(r_v) || p0 < 0 || (int64_t)p0 + M > std::numeric_limits<int>::max() || !bytes)
    return LLA_ERR_INVALID_ARG;
  *bytes = (dtype == LLA_BF16 && !prefill_absorbed_ok(d_head, r_k, r_v, 0))
               ? prefill_rebuild_bytes(B, H, d_head, p0 + M)
               : 0;
  return LLA_OK;
}

lla_status lla_prefill_attn(int dtype, int out_dtype, int B, int H, int M, int d_head, int r_k,
                            int r_v, int n_max, int p0, const void* q, const void* c_k,
                            const void* c_v, const void* u_k, const void* u_v, const void* mu_k,
                            const void* mu_v, float scale, void* out, void* workspace,
                            size_t ws_bytes, void* stream) {
  return prefill_impl(dtype, out_dtype, B, H, M, d_head, r_k, r_v, 0, 1, n_max, p0, q, nullptr,
                      c_k, c_v, nullptr, u_k, u_v, mu_k, mu_v, scale, out, workspace, ws_bytes,
                      stream);
}

lla_status lla_prefill_attn_rope(int dtype, int out_dtype, int B, int H, int M, int d_head,
                                 int r_k, int r_v, int d_rope, int H_rope, int n_max, int p0,
                                 const void* q, const void* q_rope, const void* c_k,
                                 const void* c_v, const void* r_cache, const void* u_k,
                                 const void* u_v, const void* mu_k, const void* mu_v, float scale,
                                 void* out, void* stream) {
  if (d_rope < 1) return LLA_ERR_INVALID_ARG;
  return prefill_impl(dtype, out_dtype, B, H, M, d_head, r_k, r_v, d_rope, H_rope, n_max, p0, q,
                      q_rope, c_k, c_v, r_cache, u_k, u_v, mu_k, mu_v, scale, out, nullptr, 0,
                      stream);
}

lla_status lla_rope_write(int dtype, int B, int M, int H_rope, int d_rope, const void* k_rope,
                          double base, void* r_cache, int n_max, int pos0, void* stream) {
  return rope_write_impl(dtype, B, M, H_rope, d_rope, k_rope, base, r_cache, n_max, pos0, 0, 0,
                         stream);
}

lla_status lla_rope_write_ring(int dtype, int B, int M, int H_rope, int d_rope, const void* k_rope,
                               double base, void* r_cache, int n_max, int pos0, int sink,
                               int window, void* stream) {
  if (window < 1) return LLA_ERR_INVALID_ARG;
  return rope_write_impl(dtype, B, M, H_rope, d_rope, k_rope, base, r_cache, n_max, pos0, sink,
                         window, stream);
}

lla_status lla_rope_rotate(int dtype, int B, int G, int M, int d_rope, const void* x,
                           const int32_t* pos, int pos0, double base, void* y, void* stream) {
  if (!dtype_ok(dtype) || B < 1 || G < 1 || G > 65535 || M < 1 || !rope_ok(d_rope) || pos0 < 0 ||
      !std::isfinite(base) || !(base > 1.0))
    return LLA_ERR_INVALID_ARG;
  if ((int64_t)B * G * M * d_rope > (1LL << 34) || !ptr_ok(x) || !ptr_ok(y) ||
      (pos && (reinterpret_cast<uintptr_t>(pos) & 3u)))
    return LLA_ERR_INVALID_ARG;
  lla::RopeArgs a{};
  a.dtype = dtype;
  a.B = B;
  a.G = G;
  a.M = M;
  a.dr = d_rope;
  a.x = x;
  a.pos = pos;
  a.pos0 = pos0;
  a.base = base;
  a.y = y;
  return hip_status(lla::launch_rope_rotate(a, static_cast<hipStream_t>(stream)));
}

namespace {
bool rank2d_ok(int r_k, int r_v) {
  return r_k % 32 == 0 && r_v % 16 == 0 && r_k <= LLA_MAX_RANK_2D && r_v <= LLA_MAX_RANK_2D;
}
size_t ws2d_bytes(int B, int H, int r_k, int r_v, int n_ctx) {
  const size_t qt = ((size_t)B * 2 * H * r_k * sizeof(uint16_t) + 255) / 256 * 256;
  return qt + (size_t)B * lla::decode_2d_splits(B, n_ctx) * H * (size_t)(r_v + 2) * sizeof(float);
}
}  // namespace

lla_status lla_encode_2d_workspace_bytes(int B, int M, int H, int T, int d_head, int r_k, int r_v,
                                         size_t* bytes) {
  if (B < 1 || M < 1 || H < 1 || T < 1 || !head_ok(d_head) || r_k < 1 || r_v < 1 || !bytes ||
      (int64_t)T * H * d_head > (1 << 20) || (int64_t)B * M > (1 << 30))
    return LLA_ERR_INVALID_ARG;
  *bytes = lla::encode_ws_bytes(B, M, 1, T * H * d_head, r_k, r_v);
  return LLA_OK;
}

lla_status lla_encode_2d(int dtype, int B, int M, int H, int T, int d_head, int r_k, int r_v,
                         const void* x_k, const void* x_v, const void* mu_k, const void* mu_v,
                         const void* wdt_k, const void* wdt_v, void* c_k, void* c_v, int n_max,
                         int pos0, void* workspace, size_t ws_bytes, void* stream) {
  if (!dtype_ok(dtype) || B < 1 || M < 1 || H < 1 || T < 1 || !head_ok(d_head) || r_k < 1 ||
      r_v < 1 || !cap_ok(n_max) || pos0 < 0 || (int64_t)pos0 + M > n_max)
    return LLA_ERR_INVALID_ARG;
  if ((int64_t)T * H * d_head > (1 << 20) || (int64_t)B * M > (1 << 30)) return LLA_ERR_INVALID_ARG;
  if (!ptr_ok(x_k) || !ptr_ok(x_v) || !ptr_ok(wdt_k) || !ptr_ok(wdt_v) || !ptr_ok(c_k) ||
      !ptr_ok(c_v) || !opt_ptr_ok(mu_k) || !opt_ptr_ok(mu_v))
    return LLA_ERR_INVALID_ARG;
  if (dtype != LLA_BF16 || !rank2d_ok(r_k, r_v)) return LLA_ERR_UNSUPPORTED;
  lla::EncodeArgs a{};
  a.dtype = dtype;
  a.B = B;
  a.M = M;
  a.H = 1;  // one latent per token: the whole T*H*d stack is a single "head"
  a.K = T * H * d_head;
  a.r[0] = r_k;
  a.r[1] = r_v;
  a.x[0] = x_k;
  a.x[1] = x_v;
  a.mu[0] = mu_k;
  a.mu[1] = mu_v;
  a.wdt[0] = wdt_k;
  a.wdt[1] = wdt_v;
  a.c[0] = c_k;
  a.c[1] = c_v;
  a.n_max = n_max;
  a.pos0 = pos0;
  a.k_token_major = 1;
  a.ksplit = 1;
  const size_t need = lla::encode_ws_bytes(B, M, 1, a.K, r_k, r_v);
  if (workspace && need > 0) {  // split the long K over the machine
    if (!aligned16(workspace) || ws_bytes < need) return LLA_ERR_WORKSPACE;
    a.ksplit = lla::encode_ksplit(B * M, a.K);
    a.part = static_cast<float*>(workspace);
  }
  return hip_status(lla::launch_encode(a, static_cast<hipStream_t>(stream)));
}

lla_status lla_decode_2d_workspace_bytes(int B, int H, int r_k, int r_v, int n_ctx, size_t* bytes) {
  if (B < 1 || H < 1 || r_k < 1 || r_v < 1 || n_ctx < 1 || !bytes) return LLA_ERR_INVALID_ARG;
  *bytes = ws2d_bytes(B, H, r_k, r_v, n_ctx);
  return LLA_OK;
}

lla_status lla_decode_attn_2d(int dtype, int out_dtype, int B, int H, int d_head, int r_k, int r_v,
                              int n_max, int n_ctx, const int32_t* ctx_len, const void* q,
                              const void* c_k, const void* c_v, const void* u_k, const void* u_v,
                              const void* mu_k, const void* mu_v, float scale, void* out,
                              void* workspace, size_t ws_bytes, void* stream) {
  if (!dtype_ok(dtype) || !dtype_ok(out_dtype) || B < 1 || H < 1 || !head_ok(d_head) || r_k < 1 ||
      r_v < 1 || !cap_ok(n_max) || n_ctx < 1 || n_ctx > n_max || !std::isfinite(scale) ||
      !(scale > 0.f))
    return LLA_ERR_INVALID_ARG;
  if ((int64_t)B > (1 << 20)) return LLA_ERR_INVALID_ARG;
  if (!ptr_ok(q) || !ptr_ok(c_k) || !ptr_ok(c_v) || !ptr_ok(u_k) || !ptr_ok(u_v) || !ptr_ok(out) ||
      !opt_ptr_ok(mu_k) || !opt_ptr_ok(mu_v) ||
      (ctx_len && (reinterpret_cast<uintptr_t>(ctx_len) & 3u)))
    return LLA_ERR_INVALID_ARG;
  if (dtype != LLA_BF16 || H != 16 || !rank2d_ok(r_k, r_v) || !regions_ok(n_max, r_k, r_v, 0, dtype))
    return LLA_ERR_UNSUPPORTED;
  if (!workspace || !aligned16(workspace) || ws_bytes < ws2d_bytes(B, H, r_k, r_v, n_ctx))
    return LLA_ERR_WORKSPACE;
  (void)mu_k;  // q . mu_k is constant over the context: it cancels in the softmax
  lla::Decode2dArgs a{};
  a.out_dtype = out_dtype;
  a.B = B;
  a.H = H;
  a.d = d_head;
  a.rk = r_k;
  a.rv = r_v;
  a.n_max = n_max;
  a.n_ctx = n_ctx;
  a.splits = lla::decode_2d_splits(B, n_ctx);
  a.ctx_len = ctx_len;
  a.q = q;
  a.ck = c_k;
  a.cv = c_v;
  a.uk = u_k;
  a.uv = u_v;
  a.muv = mu_v;
  a.qscale = (float)((double)scale * kLog2e);
  a.out = out;
  a.qt = static_cast<uint16_t*>(workspace);
  a.part = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                    ((size_t)B * 2 * H * r_k * sizeof(uint16_t) + 255) / 256 * 256);
  return hip_status(lla::launch_decode_2d(a, static_cast<hipStream_t>(stream)));
}

lla_status lla_prefill_2d_workspace_bytes(int B, int H, int d_head, int n_keys, size_t* bytes) {
  if (B < 1 || H < 1 || !head_ok(d_head) || n_keys < 1 || !bytes) return LLA_ERR_INVALID_ARG;
  const size_t nk = ((size_t)n_keys + 63) / 64 * 64;
  *bytes = 4 * (size_t)B * H * d_head * nk;
  return LLA_OK;
}

lla_status lla_prefill_attn_2d(int dtype, int out_dtype, int B, int H, int M, int d_head, int r_k,
                               int r_v, int n_max, int p0, const void* q, const void* c_k,
                               const void* c_v, const void* u_k, const void* u_v, const void* mu_k,
                               const void* mu_v, float scale, void* out, void* workspace,
                               size_t ws_bytes, void* stream) {
  if (!dtype_ok(dtype) || !dtype_ok(out_dtype) || B < 1 || H < 1 || M < 1 || !head_ok(d_head) ||
      r_k < 1 || r_v < 1 || !cap_ok(n_max) || p0 < 0 || (int64_t)p0 + M > n_max ||
      !std::isfinite(scale) || !(scale > 0.f))
    return LLA_ERR_INVALID_ARG;
  // launch limits: the rebuild grid's y dimension is B, the attention grid's
  // y dimension the number of 256-query blocks
  if ((int64_t)B * H * M > (1 << 30) || B > 65535 || (M + 255) / 256 > 65535) return LLA_ERR_INVALID_ARG;
  if (!ptr_ok(q) || !ptr_ok(c_k) || !ptr_ok(c_v) || !ptr_ok(u_k) || !ptr_ok(u_v) || !ptr_ok(out) ||
      !opt_ptr_ok(mu_k) || !opt_ptr_ok(mu_v))
    return LLA_ERR_INVALID_ARG;
  if (dtype != LLA_BF16 || d_head != 128 || r_k % 16 || r_v % 16 || r_k > 512 || r_v > 512 ||
      !regions_ok(n_max, r_k, r_v, 0, dtype))
    return LLA_ERR_UNSUPPORTED;
  size_t need = 0;
  lla_prefill_2d_workspace_bytes(B, H, d_head, p0 + M, &need);
  if (!workspace || !aligned16(workspace) || ws_bytes < need) return LLA_ERR_WORKSPACE;
  (void)mu_k;  // q . mu_k is the same for every key of a query: it cancels in the softmax
  lla::Prefill2dArgs a{};
  a.out_dtype = out_dtype;
  a.B = B;
  a.H = H;
  a.M = M;
  a.rk = r_k;
  a.rv = r_v;
  a.n_max = n_max;
  a.p0 = p0;
  a.nk = (p0 + M + 63) / 64 * 64;
  a.q = q;
  a.ck = c_k;
  a.cv = c_v;
  a.uk = u_k;
  a.uv = u_v;
  a.muv = mu_v;
  a.qscale = (float)((double)scale * kLog2e);
  a.out = out;
  a.kh = workspace;
  a.vt = static_cast<char*>(workspace) + need / 2;
  return hip_status(lla::launch_prefill_2d(a, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
