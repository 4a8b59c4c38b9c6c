// Memory-pressure sample for the spatial controller (HorizonServe §4.4
// "Bandwidth-pressure signal"; §5 samples the GPU's memory activity once per
// scheduling step).  On MI355X the counterpart of that reading is the
// memory-controller (UMC) activity AMD SMI reports, in percent.
//
// AMD SMI enumerates GPUs in its own order, which need not match HIP's device
// numbering (and on a shared host lists GPUs this process cannot see), so the
// sample is taken from the AMD SMI processor whose PCI address (domain, bus,
// device, function) equals the HIP device's.  AMD SMI is loaded on first use,
// so the library does not depend on it at link time.
#include <dlfcn.h>
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <vector>

#include "horizon.h"
#include "plan.h"

namespace {

struct SmiGpu {
  void* handle;
  uint64_t bdf;  // amdsmi_bdf_t.as_uint: function 3 bits, device 5, bus 8, domain above
};

struct AmdSmiStatics {
  std::once_flag once;
  bool ok = false;
  std::vector<SmiGpu> gpus;
  int (*get_activity)(void*, void*) = nullptr;
};
AmdSmiStatics g_smi;

constexpr uint64_t kAmdSmiInitGpus = 1ull << 1;  // AMDSMI_INIT_AMD_GPUS

void smi_load() {
  void* h = dlopen("libamd_smi.so", RTLD_NOW | RTLD_LOCAL);
  if (!h) h = dlopen("/opt/rocm/lib/libamd_smi.so", RTLD_NOW | RTLD_LOCAL);
  if (!h) return;
  auto init = reinterpret_cast<int (*)(uint64_t)>(dlsym(h, "amdsmi_init"));
  auto sockets = reinterpret_cast<int (*)(uint32_t*, void**)>(dlsym(h, "amdsmi_get_socket_handles"));
  auto procs = reinterpret_cast<int (*)(void*, uint32_t*, void**)>(dlsym(h, "amdsmi_get_processor_handles"));
  auto get_bdf = reinterpret_cast<int (*)(void*, uint64_t*)>(dlsym(h, "amdsmi_get_gpu_device_bdf"));
  g_smi.get_activity = reinterpret_cast<int (*)(void*, void*)>(dlsym(h, "amdsmi_get_gpu_activity"));
  if (!init || !sockets || !procs || !get_bdf || !g_smi.get_activity) return;
  if (init(kAmdSmiInitGpus) != 0) return;
  uint32_t n_sock = 0;
  if (sockets(&n_sock, nullptr) != 0 || n_sock == 0) return;
  std::vector<void*> socks(n_sock);
  if (sockets(&n_sock, socks.data()) != 0) return;
  for (uint32_t s = 0; s < n_sock; ++s) {
    uint32_t n = 0;
    if (procs(socks[s], &n, nullptr) != 0 || n == 0) continue;
    std::vector<void*> p(n);
    if (procs(socks[s], &n, p.data()) != 0) continue;
    for (uint32_t i = 0; i < n; ++i) {
      uint64_t bdf = 0;
      if (get_bdf(p[i], &bdf) == 0) g_smi.gpus.push_back({p[i], bdf});
    }
  }
  g_smi.ok = !g_smi.gpus.empty();
}

// amdsmi_bdf_t packing of a PCI address.
uint64_t pack_bdf(uint64_t domain, uint64_t bus, uint64_t device, uint64_t function) {
  return (function & 7) | ((device & 31) << 3) | ((bus & 255) << 8) | (domain << 16);
}

}  // namespace

extern "C" {

hs_status hs_pressure_sample(int32_t device, double* activity) {
  hs::clear_error();
  if (!activity) return hs::fail(HS_ERR_INVALID_ARG, "output pointer is null");
  int n_dev = 0;
  if (hipGetDeviceCount(&n_dev) != hipSuccess || device < 0 || device >= n_dev)
    return hs::fail(HS_ERR_INVALID_ARG, "HIP device %d outside the %d visible devices", device, n_dev);
  int domain = 0, bus = 0, dev = 0;
  if (hipDeviceGetAttribute(&domain, hipDeviceAttributePciDomainID, device) != hipSuccess ||
      hipDeviceGetAttribute(&bus, hipDeviceAttributePciBusId, device) != hipSuccess ||
      hipDeviceGetAttribute(&dev, hipDeviceAttributePciDeviceId, device) != hipSuccess)
    return hs::fail(HS_ERR_HIP, "could not read the PCI address of HIP device %d", device);
  std::call_once(g_smi.once, smi_load);
  if (!g_smi.ok) return hs::fail(HS_ERR_UNSUPPORTED, "AMD SMI is not available");
  // HIP reports no PCI function number; a GPU's primary function is 0.
  const uint64_t want = pack_bdf(uint64_t(domain), uint64_t(bus), uint64_t(dev), 0);
  const SmiGpu* gpu = nullptr;
  for (const SmiGpu& g : g_smi.gpus)
    if (g.bdf == want) gpu = &g;
  if (!gpu)
    return hs::fail(HS_ERR_UNSUPPORTED, "no AMD SMI GPU at PCI %04x:%02x:%02x.0 (HIP device %d)", domain, bus, dev,
                    device);
  // amdsmi_engine_usage_t: gfx_activity, umc_activity, mm_activity (percent), reserved[13].
  uint32_t usage[16] = {0};
  if (g_smi.get_activity(gpu->handle, usage) != 0)
    return hs::fail(HS_ERR_UNSUPPORTED, "AMD SMI could not read the activity of HIP device %d", device);
  *activity = double(usage[1]) / 100.0;
  return HS_OK;
}

}  // extern "C"
