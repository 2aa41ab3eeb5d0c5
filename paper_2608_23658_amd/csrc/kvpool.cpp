// Elastic per-layer KV pool over the HIP virtual-memory API (the paper,
// Section 3 "Two handles, one virtual range" and "Toggle cost"; Section 4 for
// the failure modes it must survive).
//
// Each layer reserves one virtual range [base | elastic | guard]. A base
// physical handle is mapped over [0, base) for the pool's life. Commit creates
// one elastic handle per layer and maps it at [base, base + elastic); decommit
// waits for the device, unmaps and releases those handles. The range never
// moves, so a kernel given the layer pointer reads the same addresses whether
// or not the elastic slice is present. The guard granule is never mapped: a
// read past the range faults instead of landing in another layer. Mapping
// offsets into a handle must be zero on ROCm, which is why every layer owns its
// own elastic handle rather than a slice of one large handle.
//
// Access is granted over [layer start, end of the elastic mapping) after the
// elastic map, not over the elastic sub-range alone: on this ROCm a
// hipMemSetAccess whose range starts inside a reservation fails with "invalid
// argument" for some layers and not others, while a range that starts at the
// reservation start succeeds every time. Re-granting read/write on the base
// part leaves its mapping and contents untouched.

#include <hip/hip_runtime.h>

#include <chrono>
#include <new>
#include <vector>

#include "kvattn.h"
#include "abi_internal.hpp"

struct kvpool {
  int device = 0;
  int num_layers = 0;
  size_t base_bytes = 0;
  size_t elastic_bytes = 0;
  size_t gran = 0;
  size_t align = 0;          // reservation alignment and guard size
  size_t reserve_bytes = 0;
  std::vector<char*> va;
  std::vector<hipMemGenericAllocationHandle_t> base_h;
  std::vector<hipMemGenericAllocationHandle_t> elastic_h;
  bool committed = false;
  double last_create_ms = 0, last_map_ms = 0, last_access_ms = 0, last_sync_ms = 0,
         last_unmap_ms = 0;
};

namespace {

using clock_type = std::chrono::steady_clock;

// Reservations are aligned to, and guarded by, at least one 2 MiB page.
constexpr size_t kHugePage = size_t(2) << 20;

double ms_since(clock_type::time_point t0) {
  return std::chrono::duration<double, std::milli>(clock_type::now() - t0).count();
}

hipMemAllocationProp device_prop(int device) {
  hipMemAllocationProp prop = {};
  prop.type = hipMemAllocationTypePinned;
  prop.location.type = hipMemLocationTypeDevice;
  prop.location.id = device;
  return prop;
}

hipMemAccessDesc access_desc(int device) {
  hipMemAccessDesc d = {};
  d.location.type = hipMemLocationTypeDevice;
  d.location.id = device;
  d.flags = hipMemAccessFlagsProtReadWrite;
  return d;
}

// Keeps the caller's current device across a pool call.
struct DeviceScope {
  int prev = -1;
  bool ok = false;
  explicit DeviceScope(int dev) {
    if (hipGetDevice(&prev) == hipSuccess && hipSetDevice(dev) == hipSuccess) ok = true;
  }
  ~DeviceScope() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

int hip_fail(hipError_t e, const char* what) {
  (void)hipGetLastError();   // the runtime keeps the error sticky: clear it for the caller
  const int code = (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation) ? KV_ERR_OOM
                                                                               : KV_ERR_HIP;
  return kvattn::set_error(code, "%s failed: %s", what, hipGetErrorString(e));
}

// Release the elastic handles of layers [0, n): unmap those that are mapped.
void drop_elastic(kvpool* p, int n, bool mapped) {
  for (int l = 0; l < n; ++l) {
    if (mapped) (void)hipMemUnmap(p->va[l] + p->base_bytes, p->elastic_bytes);
    if (p->elastic_h[l]) (void)hipMemRelease(p->elastic_h[l]);
    p->elastic_h[l] = 0;
  }
}

void free_pool(kvpool* p) {
  for (int l = 0; l < p->num_layers; ++l) {
    if (p->base_h[l]) {
      if (p->base_bytes) (void)hipMemUnmap(p->va[l], p->base_bytes);
      (void)hipMemRelease(p->base_h[l]);
    }
    if (p->va[l]) (void)hipMemAddressFree(p->va[l], p->reserve_bytes);
  }
  delete p;
}

}  // namespace

extern "C" int kvpool_granularity(int device, size_t* bytes) {
  kvattn::clear_error();
  if (!bytes) return kvattn::set_error(KV_ERR_INVALID, "kvpool_granularity: null output");
  DeviceScope scope(device);
  if (!scope.ok) return kvattn::set_error(KV_ERR_INVALID, "kvpool_granularity: bad device %d", device);
  hipMemAllocationProp prop = device_prop(device);
  hipError_t e = hipMemGetAllocationGranularity(bytes, &prop, hipMemAllocationGranularityMinimum);
  if (e != hipSuccess) return hip_fail(e, "hipMemGetAllocationGranularity");
  return KV_OK;
}

extern "C" int kvpool_create(int device, int num_layers, size_t base_bytes_per_layer,
                             size_t elastic_bytes_per_layer, kvpool** out) {
  kvattn::clear_error();
  if (!out) return kvattn::set_error(KV_ERR_INVALID, "kvpool_create: null output");
  *out = nullptr;
  if (num_layers <= 0)
    return kvattn::set_error(KV_ERR_INVALID, "kvpool_create: num_layers %d <= 0", num_layers);
  if (base_bytes_per_layer + elastic_bytes_per_layer == 0)
    return kvattn::set_error(KV_ERR_INVALID, "kvpool_create: empty layers");
  size_t gran = 0;
  int rc = kvpool_granularity(device, &gran);
  if (rc != KV_OK) return rc;
  if (base_bytes_per_layer % gran || elastic_bytes_per_layer % gran)
    return kvattn::set_error(KV_ERR_INVALID,
                             "kvpool_create: sizes %zu / %zu are not multiples of the %zu-byte "
                             "granularity",
                             base_bytes_per_layer, elastic_bytes_per_layer, gran);
  DeviceScope scope(device);
  if (!scope.ok) return kvattn::set_error(KV_ERR_INVALID, "kvpool_create: bad device %d", device);

  kvpool* p = new (std::nothrow) kvpool;
  if (!p) return kvattn::set_error(KV_ERR_OOM, "kvpool_create: host allocation failed");
  p->device = device;
  p->num_layers = num_layers;
  p->base_bytes = base_bytes_per_layer;
  p->elastic_bytes = elastic_bytes_per_layer;
  p->gran = gran;
  p->align = gran > kHugePage ? gran : kHugePage;
  p->reserve_bytes = base_bytes_per_layer + elastic_bytes_per_layer + p->align;  // + guard
  p->va.assign(num_layers, nullptr);
  p->base_h.assign(num_layers, 0);
  p->elastic_h.assign(num_layers, 0);

  hipMemAllocationProp prop = device_prop(device);
  hipMemAccessDesc acc = access_desc(device);
  for (int l = 0; l < num_layers; ++l) {
    void* va = nullptr;
    hipError_t e = hipMemAddressReserve(&va, p->reserve_bytes, p->align, nullptr, 0);
    if (e != hipSuccess) {
      rc = hip_fail(e, "hipMemAddressReserve");
      free_pool(p);
      return rc;
    }
    p->va[l] = static_cast<char*>(va);
    if (p->base_bytes == 0) continue;
    e = hipMemCreate(&p->base_h[l], p->base_bytes, &prop, 0);
    if (e != hipSuccess) {
      p->base_h[l] = 0;
      rc = hip_fail(e, "hipMemCreate(base)");
      free_pool(p);
      return rc;
    }
    e = hipMemMap(p->va[l], p->base_bytes, 0, p->base_h[l], 0);
    if (e != hipSuccess) {
      rc = hip_fail(e, "hipMemMap(base)");
      (void)hipMemRelease(p->base_h[l]);
      p->base_h[l] = 0;
      free_pool(p);
      return rc;
    }
    e = hipMemSetAccess(p->va[l], p->base_bytes, &acc, 1);
    if (e != hipSuccess) {
      rc = hip_fail(e, "hipMemSetAccess(base)");
      free_pool(p);   // layer l is mapped: free_pool unmaps and releases it
      return rc;
    }
  }
  *out = p;
  return KV_OK;
}

extern "C" int kvpool_layer_ptr(const kvpool* p, int layer, void** ptr) {
  kvattn::clear_error();
  if (!p || !ptr) return kvattn::set_error(KV_ERR_INVALID, "kvpool_layer_ptr: null argument");
  if (layer < 0 || layer >= p->num_layers)
    return kvattn::set_error(KV_ERR_INVALID, "kvpool_layer_ptr: layer %d outside [0, %d)",
                             layer, p->num_layers);
  *ptr = p->va[layer];
  return KV_OK;
}

extern "C" int kvpool_is_committed(const kvpool* p) {
  if (!p) return kvattn::set_error(KV_ERR_INVALID, "kvpool_is_committed: null pool");
  return p->committed ? 1 : 0;
}

extern "C" int kvpool_sizes(const kvpool* p, int* num_layers, size_t* base, size_t* elastic) {
  kvattn::clear_error();
  if (!p) return kvattn::set_error(KV_ERR_INVALID, "kvpool_sizes: null pool");
  if (num_layers) *num_layers = p->num_layers;
  if (base) *base = p->base_bytes;
  if (elastic) *elastic = p->elastic_bytes;
  return KV_OK;
}

extern "C" int kvpool_commit_elastic(kvpool* p, double* elapsed_ms) {
  kvattn::clear_error();
  const auto t0 = clock_type::now();
  if (!p) return kvattn::set_error(KV_ERR_INVALID, "kvpool_commit_elastic: null pool");
  if (p->committed || p->elastic_bytes == 0) {
    if (elapsed_ms) *elapsed_ms = ms_since(t0);
    return KV_OK;
  }
  DeviceScope scope(p->device);
  if (!scope.ok) return kvattn::set_error(KV_ERR_HIP, "kvpool_commit_elastic: hipSetDevice failed");
  hipMemAllocationProp prop = device_prop(p->device);
  hipMemAccessDesc acc = access_desc(p->device);
  // Physical allocation first: if it cannot be had, nothing was mapped.
  for (int l = 0; l < p->num_layers; ++l) {
    hipError_t e = hipMemCreate(&p->elastic_h[l], p->elastic_bytes, &prop, 0);
    if (e != hipSuccess) {
      p->elastic_h[l] = 0;
      drop_elastic(p, l, false);
      return hip_fail(e, "hipMemCreate(elastic)");
    }
  }
  const auto t1 = clock_type::now();
  for (int l = 0; l < p->num_layers; ++l) {
    hipError_t e = hipMemMap(p->va[l] + p->base_bytes, p->elastic_bytes, 0, p->elastic_h[l], 0);
    if (e != hipSuccess) {
      for (int k = 0; k < l; ++k) (void)hipMemUnmap(p->va[k] + p->base_bytes, p->elastic_bytes);
      drop_elastic(p, p->num_layers, false);
      return hip_fail(e, "hipMemMap(elastic)");
    }
  }
  const auto t2 = clock_type::now();
  for (int l = 0; l < p->num_layers; ++l) {
    hipError_t e = hipMemSetAccess(p->va[l], p->base_bytes + p->elastic_bytes, &acc, 1);
    if (e != hipSuccess) {
      drop_elastic(p, p->num_layers, true);
      return hip_fail(e, "hipMemSetAccess(elastic)");
    }
  }
  const auto t3 = clock_type::now();
  p->committed = true;
  p->last_create_ms = std::chrono::duration<double, std::milli>(t1 - t0).count();
  p->last_map_ms = std::chrono::duration<double, std::milli>(t2 - t1).count();
  p->last_access_ms = std::chrono::duration<double, std::milli>(t3 - t2).count();
  if (elapsed_ms) *elapsed_ms = ms_since(t0);
  return KV_OK;
}

extern "C" int kvpool_decommit_elastic(kvpool* p, double* elapsed_ms) {
  kvattn::clear_error();
  const auto t0 = clock_type::now();
  if (!p) return kvattn::set_error(KV_ERR_INVALID, "kvpool_decommit_elastic: null pool");
  if (!p->committed) {
    if (elapsed_ms) *elapsed_ms = ms_since(t0);
    return KV_OK;
  }
  DeviceScope scope(p->device);
  if (!scope.ok)
    return kvattn::set_error(KV_ERR_HIP, "kvpool_decommit_elastic: hipSetDevice failed");
  // Work already enqueued may still read elastic blocks: let it finish.
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
  const auto t1 = clock_type::now();
  int rc = KV_OK;
  for (int l = 0; l < p->num_layers; ++l) {
    e = hipMemUnmap(p->va[l] + p->base_bytes, p->elastic_bytes);
    if (e != hipSuccess && rc == KV_OK) rc = hip_fail(e, "hipMemUnmap(elastic)");
    e = hipMemRelease(p->elastic_h[l]);
    if (e != hipSuccess && rc == KV_OK) rc = hip_fail(e, "hipMemRelease(elastic)");
    p->elastic_h[l] = 0;
  }
  p->committed = false;
  p->last_sync_ms = std::chrono::duration<double, std::milli>(t1 - t0).count();
  p->last_unmap_ms = ms_since(t1);
  if (elapsed_ms) *elapsed_ms = ms_since(t0);
  return rc;
}

extern "C" int kvpool_last_toggle_breakdown(const kvpool* p, double* create_ms, double* map_ms,
                                            double* access_ms, double* sync_ms,
                                            double* unmap_ms) {
  kvattn::clear_error();
  if (!p) return kvattn::set_error(KV_ERR_INVALID, "kvpool_last_toggle_breakdown: null pool");
  if (create_ms) *create_ms = p->last_create_ms;
  if (map_ms) *map_ms = p->last_map_ms;
  if (access_ms) *access_ms = p->last_access_ms;
  if (sync_ms) *sync_ms = p->last_sync_ms;
  if (unmap_ms) *unmap_ms = p->last_unmap_ms;
  return KV_OK;
}

extern "C" void kvpool_destroy(kvpool* p) {
  if (!p) return;
  DeviceScope scope(p->device);
  if (p->committed) (void)kvpool_decommit_elastic(p, nullptr);
  free_pool(p);
}

extern "C" int kvpool_time_single_handle(int device, size_t bytes, double* create_ms,
                                         double* map_ms, double* access_ms, double* release_ms) {
  kvattn::clear_error();
  size_t gran = 0;
  int rc = kvpool_granularity(device, &gran);
  if (rc != KV_OK) return rc;
  if (bytes == 0 || bytes % gran)
    return kvattn::set_error(KV_ERR_INVALID,
                             "kvpool_time_single_handle: %zu bytes is not a multiple of %zu",
                             bytes, gran);
  DeviceScope scope(device);
  if (!scope.ok) return kvattn::set_error(KV_ERR_HIP, "kvpool_time_single_handle: hipSetDevice");
  const size_t align = gran > kHugePage ? gran : kHugePage;
  void* va = nullptr;
  hipError_t e = hipMemAddressReserve(&va, bytes, align, nullptr, 0);
  if (e != hipSuccess) return hip_fail(e, "hipMemAddressReserve");
  hipMemAllocationProp prop = device_prop(device);
  hipMemAccessDesc acc = access_desc(device);
  hipMemGenericAllocationHandle_t h = 0;
  const auto t0 = clock_type::now();
  e = hipMemCreate(&h, bytes, &prop, 0);
  if (e != hipSuccess) {
    (void)hipMemAddressFree(va, bytes);
    return hip_fail(e, "hipMemCreate(single)");
  }
  const auto t1 = clock_type::now();
  e = hipMemMap(va, bytes, 0, h, 0);
  const auto t2 = clock_type::now();
  hipError_t ea = e == hipSuccess ? hipMemSetAccess(va, bytes, &acc, 1) : e;
  const auto t3 = clock_type::now();
  if (e == hipSuccess) (void)hipMemUnmap(va, bytes);
  (void)hipMemRelease(h);
  const auto t4 = clock_type::now();
  (void)hipMemAddressFree(va, bytes);
  if (e != hipSuccess) return hip_fail(e, "hipMemMap(single)");
  if (ea != hipSuccess) return hip_fail(ea, "hipMemSetAccess(single)");
  auto ms = [](clock_type::time_point a, clock_type::time_point b) {
    return std::chrono::duration<double, std::milli>(b - a).count();
  };
  if (create_ms) *create_ms = ms(t0, t1);
  if (map_ms) *map_ms = ms(t1, t2);
  if (access_ms) *access_ms = ms(t2, t3);
  if (release_ms) *release_ms = ms(t3, t4);
  return KV_OK;
}
