// GMG snapshot loader: validation, load-time precompute and one-time staging
// of the snapshot in device memory (the simulator is built once per GMG,
// Sec. 3.3.2; the per-candidate work happens in simulate.hip).
#include <algorithm>
#include <cstring>
#include <mutex>
#include <new>
#include <sstream>
#include <vector>

#include "ss_internal.h"

namespace {

using i128 = __int128;
constexpr i128 kTimeLimit = (i128)1 << 62;
constexpr i128 kSumLimit = (i128)1 << 63;

// The arrays of one device allocation at 256-byte aligned offsets: add()
// records where each goes, pack() copies them once into a buffer of the
// calling thread that its later loads reuse (a load has uploaded it before it
// returns); gaps and arrays without a source are zero.  The sources must stay
// alive until pack().
struct Packer {
  struct Part {
    const void *src;
    size_t bytes, off;
  };
  std::vector<Part> parts;
  size_t size = 0;
  size_t add(const void *src, size_t bytes) {
    const size_t off = (size + 255) & ~size_t(255);
    parts.push_back({src, bytes, off});
    size = off + bytes;
    return off;
  }
  template <class T>
  size_t add(const std::vector<T> &v) {
    return add(v.data(), v.size() * sizeof(T));
  }
  const unsigned char *pack() const {
    static thread_local std::vector<unsigned char> buf;
    if (buf.size() < size) buf.resize(size);
    size_t end = 0;
    for (const Part &p : parts) {
      if (p.off > end) std::memset(buf.data() + end, 0, p.off - end);
      if (p.bytes) {
        if (p.src) std::memcpy(buf.data() + p.off, p.src, p.bytes);
        else std::memset(buf.data() + p.off, 0, p.bytes);
      }
      end = p.off + p.bytes;
    }
    return buf.data();
  }
};

int bad(const std::string &msg) { return ss_set_error(SS_ERR_INVALID_GMG, "invalid GMG: " + msg); }

}  // namespace

namespace {
constexpr int kMaxDevices = 256;
std::mutex g_pool_mu;
hipMemPool_t g_pools[kMaxDevices] = {};
hipStream_t g_aux[kMaxDevices] = {};

// Idle scratch blocks per device, each with the event that marks its last use.
struct IdleScratch {
  void *p;
  size_t bytes;
  hipEvent_t last_use;
};
constexpr size_t kIdleBlocks = 4;
std::mutex g_scratch_mu;
std::vector<IdleScratch> g_idle[kMaxDevices];

// Frees a block after its last use, in `stream`'s order.
void free_after(const IdleScratch &b, hipStream_t stream) {
  (void)hipStreamWaitEvent(stream, b.last_use, 0);
  (void)hipFreeAsync(b.p, stream);
  (void)hipEventDestroy(b.last_use);
}

// Gives every idle scratch block of the device back to the pool (in
// `stream`'s order).
void drop_idle(int device, hipStream_t stream) {
  std::vector<IdleScratch> v;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    v.swap(g_idle[device]);
  }
  for (const IdleScratch &b : v) free_after(b, stream);
}
}  // namespace

hipStream_t ss_device_aux(int device) {
  if (device < 0 || device >= kMaxDevices) {
    ss_set_error(SS_ERR_UNSUPPORTED, "device id beyond the library's stream table");
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_pool_mu);
  if (!g_aux[device]) {
    int prev = 0;
    (void)hipGetDevice(&prev);
    hipStream_t s = nullptr;
    hipError_t e = hipSetDevice(device);
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
    (void)hipSetDevice(prev);
    if (e != hipSuccess) {
      ss_set_error(SS_ERR_DEVICE, std::string("creating the second stream: ") + hipGetErrorString(e));
      return nullptr;
    }
    g_aux[device] = s;
  }
  return g_aux[device];
}

hipMemPool_t ss_device_pool(int device) {
  if (device < 0 || device >= kMaxDevices) {
    ss_set_error(SS_ERR_UNSUPPORTED, "device id beyond the library's pool table");
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_pool_mu);
  if (g_pools[device]) return g_pools[device];
  hipMemPoolProps props{};
  props.allocType = hipMemAllocationTypePinned;
  props.handleTypes = hipMemHandleTypeNone;
  props.location.type = hipMemLocationTypeDevice;
  props.location.id = device;
  uint64_t keep = UINT64_MAX;  // never hand freed memory back on synchronisation
  hipMemPool_t pool = nullptr;
  hipError_t e = hipMemPoolCreate(&pool, &props);
  if (e == hipSuccess) e = hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
  if (e != hipSuccess) {
    if (pool) (void)hipMemPoolDestroy(pool);
    ss_set_error(SS_ERR_DEVICE, std::string("creating the scratch pool: ") + hipGetErrorString(e));
    return nullptr;
  }
  g_pools[device] = pool;
  return pool;
}

hipError_t ss_pool_malloc(void **p, size_t bytes, hipMemPool_t pool, hipStream_t stream) {
  const size_t n = ss_pool_round(bytes);
  hipError_t e = hipMallocFromPoolAsync(p, n, pool, stream);
  if (e != hipErrorOutOfMemory) return e;
  (void)hipGetLastError();
  int device = -1;
  {
    std::lock_guard<std::mutex> lock(g_pool_mu);
    for (int d = 0; d < kMaxDevices && device < 0; ++d)
      if (g_pools[d] == pool) device = d;
  }
  if (device >= 0) drop_idle(device, stream);
  if (hipStreamSynchronize(stream) == hipSuccess && hipMemPoolTrimTo(pool, 0) == hipSuccess)
    e = hipMallocFromPoolAsync(p, n, pool, stream);
  if (e != hipSuccess) (void)hipGetLastError();
  return e;
}

int64_t ss_scratch_budget(int device, hipMemPool_t pool, int64_t cap, int eighths) {
  size_t free_b = 0, total_b = 0;
  if (hipMemGetInfo(&free_b, &total_b) != hipSuccess) {
    (void)hipGetLastError();
    return cap;
  }
  uint64_t reserved = 0, used = 0;
  if (pool && (hipMemPoolGetAttribute(pool, hipMemPoolAttrReservedMemCurrent, &reserved) != hipSuccess ||
               hipMemPoolGetAttribute(pool, hipMemPoolAttrUsedMemCurrent, &used) != hipSuccess)) {
    (void)hipGetLastError();
    reserved = used = 0;
  }
  size_t idle = 0;
  if (device >= 0 && device < kMaxDevices) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    for (const IdleScratch &b : g_idle[device]) idle += b.bytes;
  }
  const uint64_t avail = (uint64_t)free_b + (reserved > used ? reserved - used : 0) + idle;
  return std::min<int64_t>(cap, (int64_t)(avail / 8 * (uint64_t)eighths));
}

hipError_t ss_scratch_get(int device, hipMemPool_t pool, size_t bytes, hipStream_t stream, SsScratch *s) {
  s->p = nullptr;
  s->bytes = 0;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  IdleScratch b{};
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    std::vector<IdleScratch> &v = g_idle[device];
    int best = -1;
    for (int i = 0; i < (int)v.size(); ++i)
      if (v[i].bytes >= bytes && (best < 0 || v[i].bytes < v[best].bytes)) best = i;
    if (best >= 0) {
      b = v[best];
      v.erase(v.begin() + best);
    }
  }
  if (b.p) {
    const hipError_t e = hipStreamWaitEvent(stream, b.last_use, 0);
    if (e != hipSuccess) {
      free_after(b, stream);
      return e;
    }
    (void)hipEventDestroy(b.last_use);
    s->p = b.p;
    s->bytes = b.bytes;
    return hipSuccess;
  }
  // a quarter of headroom, so a slowly growing size finds its block again;
  // the exact size when that does not fit
  const size_t roomy = ss_pool_round(bytes + bytes / 4);
  hipError_t e = hipMallocFromPoolAsync(&s->p, roomy, pool, stream);
  if (e == hipSuccess) {
    s->bytes = roomy;
    return e;
  }
  (void)hipGetLastError();
  s->p = nullptr;
  e = ss_pool_malloc(&s->p, bytes, pool, stream);
  if (e == hipSuccess) s->bytes = ss_pool_round(bytes);
  else s->p = nullptr;
  return e;
}

hipError_t ss_scratch_put(int device, SsScratch *s, hipStream_t stream) {
  if (!s->p) return hipSuccess;
  IdleScratch b{s->p, s->bytes, nullptr};
  s->p = nullptr;
  s->bytes = 0;
  hipError_t e = hipEventCreateWithFlags(&b.last_use, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventRecord(b.last_use, stream);
  if (e != hipSuccess || device < 0 || device >= kMaxDevices) {
    if (b.last_use) (void)hipEventDestroy(b.last_use);
    const hipError_t f = hipFreeAsync(b.p, stream);
    return e != hipSuccess ? e : f;
  }
  IdleScratch out{};
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    std::vector<IdleScratch> &v = g_idle[device];
    v.push_back(b);
    if (v.size() > kIdleBlocks) {
      size_t k = 0;
      for (size_t i = 1; i < v.size(); ++i)
        if (v[i].bytes < v[k].bytes) k = i;
      out = v[k];
      v.erase(v.begin() + (ptrdiff_t)k);
    }
  }
  if (out.p) free_after(out, stream);
  return hipSuccess;
}

int ss_pool_alloc(int device, size_t bytes, hipStream_t stream, void **out) {
  *out = nullptr;
  hipMemPool_t pool = ss_device_pool(device);
  if (!pool) return SS_ERR_DEVICE;
  hipError_t e = ss_pool_malloc(out, bytes, pool, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) {
    if (*out) (void)hipFreeAsync(*out, stream);
    *out = nullptr;
    return ss_set_error(e == hipErrorOutOfMemory ? SS_ERR_OOM : SS_ERR_DEVICE,
                        std::string("allocating from the scratch pool: ") + hipGetErrorString(e));
  }
  return SS_OK;
}

void ss_pool_free(void *p, hipStream_t stream) {
  if (p) (void)hipFreeAsync(p, stream);
}

extern "C" int ss_release_cached_memory(void) {
  ss_clear_error();
  std::lock_guard<std::mutex> lock(g_pool_mu);
  int prev = 0;
  (void)hipGetDevice(&prev);
  int rc = SS_OK;
  for (int d = 0; d < kMaxDevices; ++d) {
    if (!g_pools[d]) continue;
    hipError_t e = hipSetDevice(d);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e == hipSuccess && g_aux[d]) {
      drop_idle(d, g_aux[d]);
      e = hipStreamSynchronize(g_aux[d]);
    }
    if (e == hipSuccess) e = hipMemPoolTrimTo(g_pools[d], 0);
    if (e != hipSuccess && rc == SS_OK)
      rc = ss_set_error(SS_ERR_DEVICE, std::string("trimming a scratch pool: ") + hipGetErrorString(e));
  }
  (void)hipSetDevice(prev);
  return rc;
}

extern "C" int ss_gmg_load(const ss_gmg_desc *d, ss_gmg **out) {
  ss_clear_error();
  if (!out) return ss_set_error(SS_ERR_INVALID_ARG, "ss_gmg_load: out is NULL");
  *out = nullptr;
  if (!d) return ss_set_error(SS_ERR_INVALID_ARG, "ss_gmg_load: desc is NULL");
  const int64_t N = d->n_ops, E = d->n_edges, D = d->n_dev, C = d->n_class, K = d->n_link, R = d->n_req;
  if (N < 0 || E < 0 || N >= INT32_MAX || E >= INT32_MAX) return bad("n_ops and n_edges must be in [0, 2^31-1)");
  if (D < 1 || D > 255) return bad("n_dev must be in [1, 255]");
  if (C < 1 || C > INT32_MAX || K < 1 || K > 256 || R < 0 || R >= INT32_MAX) return bad("bad n_class, n_link or n_req");
  if (N > 0 && R < 1) return bad("ops need at least one request");
  if (!d->pred_ptr || (E > 0 && !d->pred_idx) || (N > 0 && (!d->op_req || !d->dur || !d->out_bytes)) ||
      !d->dev_class || !d->link_class || !d->bw || !d->lat || !d->slice_ptr || !d->slice_begin || !d->slice_end ||
      !d->cap || (R > 0 && (!d->release || !d->deadline)))
    return ss_set_error(SS_ERR_INVALID_ARG, "ss_gmg_load: a required array is NULL");

  try {
    // ------------------------------------------------------------------ DAG
    if (d->pred_ptr[0] != 0 || d->pred_ptr[N] != E) return bad("pred_ptr must start at 0 and end at n_edges");
    for (int64_t v = 0; v < N; ++v)
      if (d->pred_ptr[v + 1] < d->pred_ptr[v] || d->pred_ptr[v + 1] > E) return bad("pred_ptr must be non-decreasing");
    std::vector<int32_t> outdeg(N, 0);
    for (int64_t v = 0; v < N; ++v) {
      const int64_t a = d->pred_ptr[v], b = d->pred_ptr[v + 1];
      if (b < a) return bad("pred_ptr must be non-decreasing");
      for (int64_t e = a; e < b; ++e) {
        const int64_t u = d->pred_idx[e];
        if (u < 0 || u >= v) {
          std::ostringstream m;
          m << "edge " << u << " -> " << v << " breaks the topological index order";
          return bad(m.str());
        }
        if (e > a && u <= d->pred_idx[e - 1]) return bad("predecessors of an op must be strictly increasing");
        outdeg[u]++;
      }
      if (d->op_req[v] < 0 || d->op_req[v] >= R) return bad("op_req out of range");
      for (int64_t c = 0; c < C; ++c)
        if (d->dur[v * C + c] < 1) return bad("durations must be >= 1");
      if (d->out_bytes[v] < 0) return bad("out_bytes must be >= 0");
    }
    // ------------------------------------------------------------ devices
    for (int64_t x = 0; x < D; ++x)
      if (d->dev_class[x] < 0 || d->dev_class[x] >= C) return bad("dev_class out of range");
    for (int64_t s = 0; s < D; ++s)
      for (int64_t t = 0; t < D; ++t)
        if (s != t && d->link_class[s * D + t] >= K) return bad("link_class out of range");
    for (int64_t k = 0; k < K; ++k)
      if (d->bw[k] < 1 || d->lat[k] < 0) return bad("bandwidth must be >= 1 and latency >= 0");
    if (d->slice_ptr[0] != 0) return bad("slice_ptr must start at 0");
    int64_t max_slices = 0;
    i128 last_start = 0;
    for (int64_t x = 0; x < D; ++x) {
      const int64_t a = d->slice_ptr[x], b = d->slice_ptr[x + 1];
      if (b <= a) return bad("every device needs at least one idle slice");
      if (b - a > 65535) return ss_set_error(SS_ERR_UNSUPPORTED, "more than 65535 idle slices on one device");
      max_slices = std::max(max_slices, b - a);
      for (int64_t k = a; k < b; ++k) {
        const int64_t s0 = d->slice_begin[k], s1 = d->slice_end[k];
        if (s0 < 0 || s0 >= s1) return bad("idle slices need 0 <= begin < end");
        if (k + 1 < b && (s1 == SS_TIME_INF || s1 > d->slice_begin[k + 1]))
          return bad("idle slices must be sorted, disjoint and finite except the last");
        if (k + 1 == b && s1 != SS_TIME_INF) return bad("the last idle slice of a device must be open (SS_TIME_INF)");
      }
      last_start = std::max<i128>(last_start, d->slice_begin[b - 1]);
    }
    for (int64_t x = 0; x < D; ++x)
      if (d->cap[x] < 0) return bad("capacity must be >= 0");
    i128 max_rel = 0;
    for (int64_t r = 0; r < R; ++r) {
      if (d->release[r] < 0) return bad("release times must be >= 0");
      if (d->deadline[r] >= ((int64_t)1 << 62) || d->deadline[r] <= -((int64_t)1 << 62))
        return bad("deadline magnitude must be below 2^62");
      max_rel = std::max<i128>(max_rel, d->release[r]);
    }
    // a running schedule's state: done ops (their predecessors done and
    // finished strictly earlier, themselves strictly after their issue),
    // issue times, the snapshot's timestamp; the latest of them bounds the
    // horizon's start like a release
    const bool snapshot = d->done_fin || d->issue_at || d->t_now != 0;
    if (d->t_now < 0 || d->t_now >= kTimeLimit) return bad("t_now must be in [0, 2^62)");
    max_rel = std::max<i128>(max_rel, d->t_now);
    for (int64_t v = 0; v < N; ++v) {
      if (d->issue_at) {
        if (d->issue_at[v] < 0 || d->issue_at[v] >= kTimeLimit) return bad("issue times must be in [0, 2^62)");
        max_rel = std::max<i128>(max_rel, d->issue_at[v]);
      }
      if (!d->done_fin || d->done_fin[v] == -1) continue;
      const int64_t f = d->done_fin[v];
      if (f < 0 || f >= kTimeLimit) return bad("done_fin must be -1 (not done) or in [0, 2^62)");
      if (d->issue_at && f <= d->issue_at[v]) return bad("a done op must finish after its issue time");
      for (int64_t e = d->pred_ptr[v]; e < d->pred_ptr[v + 1]; ++e) {
        const int64_t fu = d->done_fin[d->pred_idx[e]];
        if (fu < 0) return bad("a done op's predecessors must be done");
        if (fu >= f) return bad("a done op must finish after its predecessors");
      }
      max_rel = std::max<i128>(max_rel, f);
    }

    // ------------------------------------------- precompute + overflow bound
    std::vector<int64_t> xfer((size_t)N * K);
    i128 horizon = last_start + max_rel, bytes_total = 0;
    for (int64_t v = 0; v < N; ++v) {
      int64_t wmax = 0, xmax = 0;
      for (int64_t c = 0; c < C; ++c) wmax = std::max(wmax, d->dur[v * C + c]);
      for (int64_t k = 0; k < K; ++k) {
        const i128 x = (i128)d->lat[k] + ((i128)d->out_bytes[v] + d->bw[k] - 1) / d->bw[k];
        if (x >= kTimeLimit) return bad("transfer estimate overflows the time horizon");
        xfer[v * K + k] = (int64_t)x;
        xmax = std::max<int64_t>(xmax, (int64_t)x);
      }
      horizon += (i128)wmax + (i128)(outdeg[v] + 1) * xmax;
      bytes_total += d->out_bytes[v];
      if (horizon >= kTimeLimit) return bad("time horizon bound reaches 2^62");
      if (bytes_total * (D + 1) >= kSumLimit) return bad("total tensor bytes times (n_dev + 1) reaches 2^63");
    }
    if (horizon * (i128)std::max<int64_t>(N, 1) >= kSumLimit) return bad("n_ops times the horizon reaches 2^63");

    // successor CSR, ascending within each op
    std::vector<int32_t> succ_ptr(N + 1, 0), succ_idx(E), succ_pe(E), fill(N, 0);
    for (int64_t v = 0; v < N; ++v) succ_ptr[v + 1] = succ_ptr[v] + outdeg[v];
    for (int64_t v = 0; v < N; ++v)
      for (int64_t e = d->pred_ptr[v]; e < d->pred_ptr[v + 1]; ++e) {
        const int32_t u = d->pred_idx[e];
        succ_pe[succ_ptr[u] + fill[u]] = (int32_t)e;
        succ_idx[succ_ptr[u] + fill[u]++] = (int32_t)v;
      }
    std::vector<int32_t> pred_ptr(d->pred_ptr, d->pred_ptr + N + 1), slice_ptr(D + 1);
    for (int64_t x = 0; x <= D; ++x) slice_ptr[x] = (int32_t)d->slice_ptr[x];
    const int64_t S = d->slice_ptr[D];
    if (S >= INT32_MAX) return ss_set_error(SS_ERR_UNSUPPORTED, "too many idle slices in total");

    // 32-bit time path: every time the simulation can produce is <= horizon
    int64_t max_bytes = 0;
    for (int64_t v = 0; v < N; ++v) max_bytes = std::max(max_bytes, d->out_bytes[v]);
    const bool time32 = !snapshot && horizon < (i128)UINT32_MAX && N <= 65535 && E <= 65535 && max_slices <= 65535 &&
                        max_bytes <= (int64_t)UINT32_MAX;
    std::vector<uint32_t> dur32, xfer32, sb32, se32, rel32, meta, lbits, bytes32, succ2, succ2_pe, lutk, lutw;
    std::vector<uint8_t> lgrp;
    // ready-time dispatch: the ops without predecessors by (release of their
    // request, index); on the 32-bit path also as keys release << 16 | op
    std::vector<int32_t> src_ops;
    for (int64_t v = 0; v < N; ++v)
      if (d->pred_ptr[v + 1] == d->pred_ptr[v]) src_ops.push_back((int32_t)v);
    std::stable_sort(src_ops.begin(), src_ops.end(),
                     [&](int32_t a, int32_t b) { return d->release[d->op_req[a]] < d->release[d->op_req[b]]; });
    std::vector<uint64_t> src_keys;
    if (time32)
      for (const int32_t v : src_ops) src_keys.push_back((uint64_t)d->release[d->op_req[v]] << 16 | (uint64_t)v);
    int32_t lsame = 0, lshift = -1;
    int64_t lut_nb = 0, lut_shift = 0;
    int64_t max_outdeg = 0;
    for (int64_t v = 0; v < N; ++v) max_outdeg = std::max<int64_t>(max_outdeg, outdeg[v]);
    const int64_t lwords = (D + 31) / 32;
    // 32-bit byte sums in the peak pass: with every size divided by their
    // common power of two, what can be live on one device at once (each output
    // and at most one copy per consumer edge) sums below 2^32
    int32_t pshift = 0, pnarrow = 0;
    if (time32) {
      uint64_t any_bits = 0;
      for (int64_t v = 0; v < N; ++v) any_bits |= (uint64_t)d->out_bytes[v];
      pshift = any_bits ? __builtin_ctzll(any_bits) : 0;
      i128 total = 0;
      for (int64_t v = 0; v < N; ++v) total += (i128)(d->out_bytes[v] >> pshift) * (1 + outdeg[v]);
      pnarrow = total < ((i128)1 << 32) ? 1 : 0;
    }
    const int64_t meta_stride = std::max<int64_t>(128, (N + 63) / 64 * 64 + 64);  // two blocks of 64 past any op
    if (time32) {
      meta.assign((size_t)kOpMetaFields * meta_stride, 0);
      auto M = [&](int f, int64_t v) -> uint32_t & { return meta[(size_t)f * meta_stride + v]; };
      for (int64_t v = 0; v < N; ++v) {
        const int64_t e0 = d->pred_ptr[v], np = d->pred_ptr[v + 1] - e0;
        M(kMetaDur, v) = C == 1 ? (uint32_t)d->dur[v] : 0u;
        M(kMetaReq, v) = (uint32_t)d->op_req[v] | (uint32_t)std::min<int64_t>(np, 0xFFFF) << 16;
        M(kMetaRel, v) = (uint32_t)d->release[d->op_req[v]];
        uint32_t p[4] = {0xFFFFu, 0xFFFFu, 0xFFFFu, 0xFFFFu};
        for (int64_t i = 0; i < std::min<int64_t>(np, 4); ++i) {
          const int64_t u = d->pred_idx[e0 + i];
          p[i] = (uint32_t)u;
          for (int64_t k = 0; k < 2; ++k) M(kMetaX + 2 * (int)i + (int)k, v) = (uint32_t)xfer[u * K + std::min<int64_t>(k, K - 1)];
        }
        M(kMetaP01, v) = p[0] | p[1] << 16;
        M(kMetaP23, v) = p[2] | p[3] << 16;
        M(kMetaE0, v) = (uint32_t)e0;
      }
      dur32.assign(d->dur, d->dur + N * C);
      bytes32.assign(d->out_bytes, d->out_bytes + N);
      if (max_outdeg <= 2) {
        succ2.assign(N, 0xFFFFFFFFu);
        for (int64_t v = 0; v < N; ++v)
          for (int64_t q = 0; q < outdeg[v]; ++q) {
            const uint32_t x = (uint32_t)succ_idx[succ_ptr[v] + q];
            succ2[v] = q == 0 ? (0xFFFF0000u | x) : ((succ2[v] & 0xFFFFu) | x << 16);
          }
        if (E < 0xFFFF) {
          succ2_pe.assign(N, 0xFFFFFFFFu);
          for (int64_t v = 0; v < N; ++v)
            for (int64_t q = 0; q < outdeg[v]; ++q) {
              const uint32_t pe = (uint32_t)succ_pe[succ_ptr[v] + q];
              succ2_pe[v] = q == 0 ? (0xFFFF0000u | pe) : ((succ2_pe[v] & 0xFFFFu) | pe << 16);
            }
        }
      }
      if (K <= 2) {
        // device groups: join devices linked by class `same`, then check that
        // every distinct pair's class is `same` exactly within a group
        for (int same = 0; same < 2 && lgrp.empty(); ++same) {
          std::vector<int64_t> root(D);
          for (int64_t a = 0; a < D; ++a) root[a] = a;
          auto find = [&](int64_t a) {
            while (root[a] != a) a = root[a] = root[root[a]];
            return a;
          };
          for (int64_t a = 0; a < D; ++a)
            for (int64_t b = 0; b < D; ++b)
              if (a != b && d->link_class[a * D + b] == same) root[find(a)] = find(b);
          std::vector<int64_t> id(D, -1);
          std::vector<uint8_t> grp(D);
          int64_t ng = 0;
          for (int64_t a = 0; a < D; ++a) {
            const int64_t r = find(a);
            if (id[r] < 0) id[r] = ng++;
            grp[a] = (uint8_t)id[r];
          }
          bool ok = ng <= 256;
          for (int64_t a = 0; a < D && ok; ++a)
            for (int64_t b = 0; b < D && ok; ++b)
              if (a != b) ok = (d->link_class[a * D + b] == same) == (grp[a] == grp[b]);
          if (ok) {
            lgrp = grp;
            lsame = same;
            for (int s = 0; s < 8 && lshift < 0; ++s) {
              bool pow2 = true;
              for (int64_t a = 0; a < D && pow2; ++a) pow2 = grp[a] == (a >> s);
              if (pow2) lshift = s;
            }
          }
        }
        lbits.assign((size_t)D * lwords, 0u);
        for (int64_t a = 0; a < D; ++a)
          for (int64_t b = 0; b < D; ++b)
            if (d->link_class[a * D + b]) lbits[a * lwords + b / 32] |= 1u << (b % 32);
      }
      xfer32.assign(xfer.begin(), xfer.end());
      rel32.assign(d->release, d->release + R);
      sb32.assign(S + 1, UINT32_MAX);  // spare entry: read ahead, never used
      se32.assign(S + 1, UINT32_MAX);

      for (int64_t k = 0; k < S; ++k) {
        sb32[k] = (uint32_t)d->slice_begin[k];
        se32[k] = d->slice_end[k] == SS_TIME_INF ? UINT32_MAX : (uint32_t)d->slice_end[k];
      }
      // time -> slice lookup: about 128K buckets in all (at least 64 per device)
      uint32_t max_end = 0;
      for (int64_t k = 0; k < S; ++k)
        if (se32[k] != UINT32_MAX) max_end = std::max(max_end, se32[k]);
      const int64_t nb_target = std::max<int64_t>(64, 131072 / D);
      while (((int64_t)max_end >> lut_shift) + 2 > nb_target) ++lut_shift;
      lut_nb = ((int64_t)max_end >> lut_shift) + 2;
      lutk.assign((size_t)D * lut_nb, 0u);
      lutw.assign((size_t)D * lut_nb * 4, UINT32_MAX);
      for (int64_t x = 0; x < D; ++x) {
        const int64_t a = d->slice_ptr[x], b = d->slice_ptr[x + 1];
        int64_t k = 0;
        for (int64_t bk = 0; bk < lut_nb; ++bk) {
          const uint64_t t0 = (uint64_t)bk << lut_shift;
          while (a + k < b - 1 && (uint64_t)se32[a + k] < t0) ++k;  // the last slice is open
          const size_t e = (size_t)(x * lut_nb + bk);
          lutk[e] = (uint32_t)k;
          lutw[4 * e] = sb32[a + k];
          lutw[4 * e + 1] = se32[a + k];
          lutw[4 * e + 2] = sb32[a + k + 1];  // spare entry past the last slice
          lutw[4 * e + 3] = se32[a + k + 1];
        }
      }
    }

    // ------------------------------------------------------------- staging
    Packer pk;
    const size_t o_pred_ptr = pk.add(pred_ptr);
    const size_t o_pred_idx = pk.add(d->pred_idx, E * sizeof(int32_t));
    const size_t o_succ_ptr = pk.add(succ_ptr);
    const size_t o_succ_idx = pk.add(succ_idx);
    const size_t o_succ_pe = pk.add(succ_pe);
    const size_t o_op_req = pk.add(d->op_req, N * sizeof(int32_t));
    const size_t o_dev_class = pk.add(d->dev_class, D * sizeof(int32_t));
    const size_t o_slice_ptr = pk.add(slice_ptr);
    const size_t o_dur = pk.add(d->dur, N * C * sizeof(int64_t));
    const size_t o_bytes = pk.add(d->out_bytes, N * sizeof(int64_t));
    const size_t o_xfer = pk.add(xfer);
    const size_t o_sb = pk.add(d->slice_begin, S * sizeof(int64_t));
    const size_t o_se = pk.add(d->slice_end, S * sizeof(int64_t));
    const size_t o_cap = pk.add(d->cap, D * sizeof(int64_t));
    const size_t o_rel = pk.add(d->release, R * sizeof(int64_t));
    const size_t o_dl = pk.add(d->deadline, R * sizeof(int64_t));
    const size_t o_link = pk.add(d->link_class, D * D);
    const size_t o_done = d->done_fin ? pk.add(d->done_fin, N * sizeof(int64_t)) : 0;
    const size_t o_issue = d->issue_at ? pk.add(d->issue_at, N * sizeof(int64_t)) : 0;
    const size_t o_dur32 = pk.add(dur32), o_xfer32 = pk.add(xfer32), o_sb32 = pk.add(sb32), o_se32 = pk.add(se32),
                 o_rel32 = pk.add(rel32), o_meta = pk.add(meta), o_lbits = pk.add(lbits), o_b32 = pk.add(bytes32),
                 o_succ2 = pk.add(succ2), o_succ2_pe = pk.add(succ2_pe), o_lutk = pk.add(lutk), o_lutw = pk.add(lutw), o_lgrp = pk.add(lgrp),
                 o_src = pk.add(src_keys), o_src_ops = pk.add(src_ops);
    pk.add(nullptr, 256);  // tail padding

    ss_gmg *g = new ss_gmg();
    if (hipGetDevice(&g->device) != hipSuccess) {
      delete g;
      return ss_set_error(SS_ERR_DEVICE, "hipGetDevice failed");
    }
    g->aux = ss_device_aux(g->device);
    g->pool = g->aux ? ss_device_pool(g->device) : nullptr;
    const unsigned char *packed = pk.pack();
    int arc = g->pool ? ss_pool_alloc(g->device, pk.size, g->aux, &g->dev_mem) : SS_ERR_DEVICE;
    hipError_t e = hipSuccess;
    if (arc == SS_OK) {
      e = hipMemcpyAsync(g->dev_mem, packed, pk.size, hipMemcpyHostToDevice, g->aux);
      if (e == hipSuccess) e = hipStreamSynchronize(g->aux);
      if (e != hipSuccess) arc = ss_set_error(SS_ERR_DEVICE, "copying the staged GMG failed");
    }
    if (arc != SS_OK) {
      if (g->aux) {
        ss_pool_free(g->dev_mem, g->aux);
        (void)hipStreamSynchronize(g->aux);
      }
      delete g;
      return arc;
    }
    auto *base = static_cast<unsigned char *>(g->dev_mem);
    GmgView &V = g->view;
    V.n_ops = (int32_t)N;
    V.n_dev = (int32_t)D;
    V.n_class = (int32_t)C;
    V.n_link = (int32_t)K;
    V.n_req = (int32_t)R;
    V.pred_ptr = reinterpret_cast<const int32_t *>(base + o_pred_ptr);
    V.pred_idx = reinterpret_cast<const int32_t *>(base + o_pred_idx);
    V.succ_ptr = reinterpret_cast<const int32_t *>(base + o_succ_ptr);
    V.succ_idx = reinterpret_cast<const int32_t *>(base + o_succ_idx);
    V.succ_pe = reinterpret_cast<const int32_t *>(base + o_succ_pe);
    V.op_req = reinterpret_cast<const int32_t *>(base + o_op_req);
    V.dev_class = reinterpret_cast<const int32_t *>(base + o_dev_class);
    V.slice_ptr = reinterpret_cast<const int32_t *>(base + o_slice_ptr);
    V.dur = reinterpret_cast<const int64_t *>(base + o_dur);
    V.out_bytes = reinterpret_cast<const int64_t *>(base + o_bytes);
    V.xfer = reinterpret_cast<const int64_t *>(base + o_xfer);
    V.slice_begin = reinterpret_cast<const int64_t *>(base + o_sb);
    V.slice_end = reinterpret_cast<const int64_t *>(base + o_se);
    V.cap = reinterpret_cast<const int64_t *>(base + o_cap);
    V.release = reinterpret_cast<const int64_t *>(base + o_rel);
    V.deadline = reinterpret_cast<const int64_t *>(base + o_dl);
    V.link_class = reinterpret_cast<const uint8_t *>(base + o_link);
    V.done_fin = d->done_fin ? reinterpret_cast<const int64_t *>(base + o_done) : nullptr;
    V.issue_at = d->issue_at ? reinterpret_cast<const int64_t *>(base + o_issue) : nullptr;
    V.t_now = d->t_now;
    V.time32 = time32 ? 1 : 0;
    V.dur32 = reinterpret_cast<const uint32_t *>(base + o_dur32);
    V.xfer32 = reinterpret_cast<const uint32_t *>(base + o_xfer32);
    V.slice_begin32 = reinterpret_cast<const uint32_t *>(base + o_sb32);
    V.slice_end32 = reinterpret_cast<const uint32_t *>(base + o_se32);
    V.release32 = reinterpret_cast<const uint32_t *>(base + o_rel32);
    V.op_meta = reinterpret_cast<const uint32_t *>(base + o_meta);
    V.meta_stride = (int32_t)meta_stride;
    V.link_bits = lbits.empty() ? nullptr : reinterpret_cast<const uint32_t *>(base + o_lbits);
    V.link_words = (int32_t)lwords;
    V.bytes32 = reinterpret_cast<const uint32_t *>(base + o_b32);
    V.peak_shift = pshift;
    V.peak_narrow = pnarrow;
    V.succ2 = succ2.empty() ? nullptr : reinterpret_cast<const uint32_t *>(base + o_succ2);
    V.succ2_pe = succ2_pe.empty() ? nullptr : reinterpret_cast<const uint32_t *>(base + o_succ2_pe);
    V.link_grp = lgrp.empty() ? nullptr : reinterpret_cast<const uint8_t *>(base + o_lgrp);
    V.src_keys = reinterpret_cast<const uint64_t *>(base + o_src);
    V.src_ops = reinterpret_cast<const int32_t *>(base + o_src_ops);
    V.n_src = (int32_t)src_ops.size();
    V.link_same = lsame;
    V.link_shift = lshift;
    V.lut_k = reinterpret_cast<const uint32_t *>(base + o_lutk);
    V.lut_w = reinterpret_cast<const uint4 *>(base + o_lutw);
    V.lut_nb = (int32_t)lut_nb;
    V.lut_shift = (int32_t)lut_shift;
    g->n_ops = N;
    g->n_edges = E;
    g->n_dev = D;
    g->n_class = C;
    g->n_link = K;
    g->n_req = R;
    g->max_slices = max_slices;
    g->horizon = (int64_t)horizon;
    g->snapshot = snapshot;
    for (int64_t v = 0; v < N; ++v) g->max_indeg = std::max<int64_t>(g->max_indeg, d->pred_ptr[v + 1] - d->pred_ptr[v]);
    g->max_outdeg = max_outdeg;
    *out = g;
    return SS_OK;
  } catch (const std::bad_alloc &) {
    return ss_set_error(SS_ERR_OOM, "host allocation failed while loading the GMG");
  }
}

extern "C" void ss_gmg_free(ss_gmg *g) {
  if (!g) return;
  int prev = 0;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(g->device);
  (void)hipDeviceSynchronize();
  ss_pool_free(g->dev_mem, g->aux);
  (void)hipStreamSynchronize(g->aux);
  (void)hipSetDevice(prev);
  delete g;
}

extern "C" int ss_gmg_info(const ss_gmg *g, int64_t *n_ops, int64_t *n_dev, int64_t *n_req) {
  ss_clear_error();
  if (!g) return ss_set_error(SS_ERR_INVALID_ARG, "ss_gmg_info: g is NULL");
  if (n_ops) *n_ops = g->n_ops;
  if (n_dev) *n_dev = g->n_dev;
  if (n_req) *n_req = g->n_req;
  return SS_OK;
}
