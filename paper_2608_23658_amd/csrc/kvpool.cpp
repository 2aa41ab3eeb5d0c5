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
  // Committed through one whole handle per layer over base + elastic (the
  // naive toggle): whole_h holds those handles and base_h is empty.
  std::vector<hipMemGenericAllocationHandle_t> whole_h;
  bool committed = false;
  bool whole = false;
  kvpool_steps last;   // host wall time of each step of the last commit / decommit
};

namespace {

using clock_type = std::chrono::steady_clock;

// Reservations are aligned to, and guarded by, at least one 2 MiB page.
constexpr size_t kHugePage = size_t(2) << 20;

double ms_since(clock_type::time_point t0) {
  return std::chrono::duration<double, std::milli>(clock_type::now() - t0).count();
}

double ms_between(clock_type::time_point a, clock_type::time_point b) {
  return std::chrono::duration<double, std::milli>(b - a).count();
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
    if (!p->whole_h.empty() && p->whole_h[l]) {
      (void)hipMemUnmap(p->va[l], p->base_bytes + p->elastic_bytes);
      (void)hipMemRelease(p->whole_h[l]);
    }
    if (p->va[l]) (void)hipMemAddressFree(p->va[l], p->reserve_bytes);
  }
  delete p;
}

// Staging ranges: one reserved range per layer, each mapped to a new handle
// so that the layer's current contents can be copied into it before the
// handles are swapped under the layer's own range.
struct Staging {
  std::vector<char*> va;
  size_t bytes = 0;
  std::vector<bool> mapped;
  ~Staging() {
    for (size_t l = 0; l < va.size(); ++l) {
      if (mapped[l]) (void)hipMemUnmap(va[l], bytes);
      if (va[l]) (void)hipMemAddressFree(va[l], bytes);
    }
  }
};

// Map handles h[l] at fresh ranges of `bytes`, copy the first `copy_bytes`
// of each layer's range into them, and wait for the copies; the staging
// mappings go away with st.
int stage_and_copy(kvpool* p, const std::vector<hipMemGenericAllocationHandle_t>& h,
                   size_t bytes, size_t copy_bytes, Staging& st) {
  hipMemAccessDesc acc = access_desc(p->device);
  st.bytes = bytes;
  st.va.assign(p->num_layers, nullptr);
  st.mapped.assign(p->num_layers, false);
  for (int l = 0; l < p->num_layers; ++l) {
    void* v = nullptr;
    hipError_t e = hipMemAddressReserve(&v, bytes, p->align, nullptr, 0);
    if (e != hipSuccess) return hip_fail(e, "hipMemAddressReserve(staging)");
    st.va[l] = static_cast<char*>(v);
    e = hipMemMap(st.va[l], bytes, 0, h[l], 0);
    if (e != hipSuccess) return hip_fail(e, "hipMemMap(staging)");
    st.mapped[l] = true;
    e = hipMemSetAccess(st.va[l], bytes, &acc, 1);
    if (e != hipSuccess) return hip_fail(e, "hipMemSetAccess(staging)");
  }
  if (copy_bytes) {
    for (int l = 0; l < p->num_layers; ++l) {
      hipError_t e = hipMemcpyAsync(st.va[l], p->va[l], copy_bytes, hipMemcpyDeviceToDevice,
                                    nullptr);
      if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(staging)");
    }
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize(staging)");
  }
  return KV_OK;
}

void release_all(std::vector<hipMemGenericAllocationHandle_t>& h) {
  for (auto& x : h) {
    if (x) (void)hipMemRelease(x);
    x = 0;
  }
}

// Swap the mapping under every layer's range: [0, old_bytes) of handles
// old_h out, [0, new_bytes) of handles new_h in. On a failure every layer is
// put back on its old handle. Accumulates the unmap and map time.
int swap_mappings(kvpool* p, std::vector<hipMemGenericAllocationHandle_t>& old_h,
                  size_t old_bytes, std::vector<hipMemGenericAllocationHandle_t>& new_h,
                  size_t new_bytes, double* unmap_ms, double* map_ms) {
  hipMemAccessDesc acc = access_desc(p->device);
  auto restore_old = [&](int k) {
    if (old_bytes && hipMemMap(p->va[k], old_bytes, 0, old_h[k], 0) == hipSuccess)
      (void)hipMemSetAccess(p->va[k], old_bytes, &acc, 1);
  };
  *unmap_ms = *map_ms = 0;
  for (int l = 0; l < p->num_layers; ++l) {
    const auto t0 = clock_type::now();
    hipError_t e = old_bytes ? hipMemUnmap(p->va[l], old_bytes) : hipSuccess;
    const auto t1 = clock_type::now();
    *unmap_ms += ms_between(t0, t1);
    const bool unmapped = e == hipSuccess;
    if (unmapped) e = hipMemMap(p->va[l], new_bytes, 0, new_h[l], 0);
    *map_ms += ms_between(t1, clock_type::now());
    if (e != hipSuccess) {
      const int rc = hip_fail(e, "swapping a layer's handles");
      if (unmapped) restore_old(l);
      for (int k = 0; k < l; ++k) {
        (void)hipMemUnmap(p->va[k], new_bytes);
        restore_old(k);
      }
      (void)hipGetLastError();
      return rc;
    }
  }
  return KV_OK;
}

// The whole-handle decommit (the device is synchronised): new base handles,
// the base contents copied out of the whole handles, the handles swapped,
// the whole handles released.
int decommit_whole(kvpool* p) {
  hipMemAllocationProp prop = device_prop(p->device);
  hipMemAccessDesc acc = access_desc(p->device);
  const size_t whole = p->base_bytes + p->elastic_bytes;
  const auto t1 = clock_type::now();
  std::vector<hipMemGenericAllocationHandle_t> b(p->num_layers, 0);
  if (p->base_bytes) {
    for (int l = 0; l < p->num_layers; ++l) {
      hipError_t e = hipMemCreate(&b[l], p->base_bytes, &prop, 0);
      if (e != hipSuccess) {
        b[l] = 0;
        release_all(b);
        return hip_fail(e, "hipMemCreate(base)");
      }
    }
  }
  const auto t2 = clock_type::now();
  if (p->base_bytes) {
    Staging st;
    const int rc = stage_and_copy(p, b, p->base_bytes, p->base_bytes, st);
    if (rc != KV_OK) {
      release_all(b);
      return rc;
    }
  }
  const auto t3 = clock_type::now();
  double unmap_ms = 0, map_ms = 0;
  int rc = KV_OK;
  if (p->base_bytes) {
    rc = swap_mappings(p, p->whole_h, whole, b, p->base_bytes, &unmap_ms, &map_ms);
  } else {
    for (int l = 0; l < p->num_layers; ++l) (void)hipMemUnmap(p->va[l], whole);
  }
  if (rc != KV_OK) {
    release_all(b);
    return rc;
  }
  const auto t4 = clock_type::now();
  for (int l = 0; l < p->num_layers && p->base_bytes; ++l) {
    hipError_t e = hipMemSetAccess(p->va[l], p->base_bytes, &acc, 1);
    if (e != hipSuccess && rc == KV_OK) rc = hip_fail(e, "hipMemSetAccess(base)");
  }
  const auto t5 = clock_type::now();
  release_all(p->whole_h);
  const auto t6 = clock_type::now();
  p->base_h = b;
  p->committed = false;
  p->whole = false;
  p->last.decommit_create_ms = ms_between(t1, t2);
  p->last.decommit_copy_ms = ms_between(t2, t3);
  p->last.decommit_unmap_ms = unmap_ms;
  p->last.decommit_map_ms = ms_between(t3, t4) - unmap_ms;
  p->last.decommit_access_ms = ms_between(t4, t5);
  p->last.decommit_release_ms = ms_between(t5, t6);
  return rc;
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
  p->whole_h.assign(num_layers, 0);

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
  p->whole = false;
  p->last.commit_create_ms = ms_between(t0, t1);
  p->last.commit_copy_ms = 0;
  p->last.commit_map_ms = ms_between(t1, t2);
  p->last.commit_access_ms = ms_between(t2, t3);
  p->last.commit_release_ms = 0;
  if (elapsed_ms) *elapsed_ms = ms_since(t0);
  return KV_OK;
}

extern "C" int kvpool_commit_whole(kvpool* p, double* elapsed_ms) {
  kvattn::clear_error();
  const auto t0 = clock_type::now();
  if (!p) return kvattn::set_error(KV_ERR_INVALID, "kvpool_commit_whole: null pool");
  if (p->committed) {
    if (!p->whole)
      return kvattn::set_error(KV_ERR_STATE,
                               "kvpool_commit_whole: committed with two handles; decommit first");
    if (elapsed_ms) *elapsed_ms = ms_since(t0);
    return KV_OK;
  }
  if (p->elastic_bytes == 0) {
    if (elapsed_ms) *elapsed_ms = ms_since(t0);
    return KV_OK;
  }
  DeviceScope scope(p->device);
  if (!scope.ok) return kvattn::set_error(KV_ERR_HIP, "kvpool_commit_whole: hipSetDevice failed");
  hipMemAllocationProp prop = device_prop(p->device);
  hipMemAccessDesc acc = access_desc(p->device);
  const size_t whole = p->base_bytes + p->elastic_bytes;
  // 1. physical allocation of every layer's whole range
  std::vector<hipMemGenericAllocationHandle_t> h(p->num_layers, 0);
  for (int l = 0; l < p->num_layers; ++l) {
    hipError_t e = hipMemCreate(&h[l], whole, &prop, 0);
    if (e != hipSuccess) {
      h[l] = 0;
      release_all(h);
      return hip_fail(e, "hipMemCreate(whole)");
    }
  }
  const auto t1 = clock_type::now();
  // 2. the base contents copied into the new handles
  {
    Staging st;
    const int rc = stage_and_copy(p, h, whole, p->base_bytes, st);
    if (rc != KV_OK) {
      release_all(h);
      return rc;
    }
  }
  const auto t2 = clock_type::now();
  // 3. the layer ranges switched from the base handles to the whole handles
  double unmap_ms = 0, map_ms = 0;
  int rc = swap_mappings(p, p->base_h, p->base_bytes, h, whole, &unmap_ms, &map_ms);
  if (rc != KV_OK) {
    release_all(h);
    return rc;
  }
  const auto t3 = clock_type::now();
  for (int l = 0; l < p->num_layers; ++l) {
    hipError_t e = hipMemSetAccess(p->va[l], whole, &acc, 1);
    if (e != hipSuccess && rc == KV_OK) rc = hip_fail(e, "hipMemSetAccess(whole)");
  }
  const auto t4 = clock_type::now();
  release_all(p->base_h);
  const auto t5 = clock_type::now();
  p->whole_h = h;
  p->committed = true;
  p->whole = true;
  p->last.commit_create_ms = ms_between(t0, t1);
  p->last.commit_copy_ms = ms_between(t1, t2);
  p->last.commit_map_ms = ms_between(t2, t3);   // unmapping the base handles included
  p->last.commit_access_ms = ms_between(t3, t4);
  p->last.commit_release_ms = ms_between(t4, t5);
  if (elapsed_ms) *elapsed_ms = ms_since(t0);
  return rc;
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
  p->last.decommit_sync_ms = ms_between(t0, t1);
  if (p->whole) {
    const int rc = decommit_whole(p);
    if (elapsed_ms) *elapsed_ms = ms_since(t0);
    return rc;
  }
  int rc = KV_OK;
  for (int l = 0; l < p->num_layers; ++l) {
    e = hipMemUnmap(p->va[l] + p->base_bytes, p->elastic_bytes);
    if (e != hipSuccess && rc == KV_OK) rc = hip_fail(e, "hipMemUnmap(elastic)");
  }
  const auto t2 = clock_type::now();
  for (int l = 0; l < p->num_layers; ++l) {
    e = hipMemRelease(p->elastic_h[l]);
    if (e != hipSuccess && rc == KV_OK) rc = hip_fail(e, "hipMemRelease(elastic)");
    p->elastic_h[l] = 0;
  }
  const auto t3 = clock_type::now();
  p->committed = false;
  p->last.decommit_create_ms = p->last.decommit_copy_ms = 0;
  p->last.decommit_unmap_ms = ms_between(t1, t2);
  p->last.decommit_release_ms = ms_between(t2, t3);
  p->last.decommit_map_ms = p->last.decommit_access_ms = 0;
  if (elapsed_ms) *elapsed_ms = ms_since(t0);
  return rc;
}

extern "C" int kvpool_last_toggle_breakdown(const kvpool* p, double* create_ms, double* map_ms,
                                            double* access_ms, double* sync_ms,
                                            double* unmap_ms) {
  kvattn::clear_error();
  if (!p) return kvattn::set_error(KV_ERR_INVALID, "kvpool_last_toggle_breakdown: null pool");
  if (create_ms) *create_ms = p->last.commit_create_ms;
  if (map_ms) *map_ms = p->last.commit_map_ms;
  if (access_ms) *access_ms = p->last.commit_access_ms;
  if (sync_ms) *sync_ms = p->last.decommit_sync_ms;
  if (unmap_ms) *unmap_ms = p->last.decommit_unmap_ms + p->last.decommit_release_ms;
  return KV_OK;
}

extern "C" int kvpool_last_toggle_steps(const kvpool* p, kvpool_steps* out) {
  kvattn::clear_error();
  if (!p || !out) return kvattn::set_error(KV_ERR_INVALID, "kvpool_last_toggle_steps: null");
  *out = p->last;
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
