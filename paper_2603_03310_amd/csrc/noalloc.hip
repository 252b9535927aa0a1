// ent_entropy_temperature_noalloc: the entropy and controller entry point
// for callers that cannot allocate device memory.  It needs no context and
// allocates nothing: the only scratch its kernels use (the chunk triples of
// the entropy pass and, with an estimator, the chunk threads' logit maxima)
// lives in the file-scope device array `scratch` below, of a fixed size.
// Each GPU the library runs on holds its own copy of the array until the
// process ends.  Host code never passes the array's name to a kernel (in
// host code that name is a stand-in, not a device address): the device
// address is looked up once per device with hipGetSymbolAddress and kept.
// The kernels are those of ent_entropy_temperature, so both entry points
// give the same bits.

#include <mutex>

#include "ent_internal.h"

namespace {

static __device__ __align__(256) unsigned char scratch[ENT_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;

// Per device: the array's device address and the launch facts the entropy
// pass needs (compute units, resident workgroups of the chunk pass at each
// head dimension), looked up on the first call with that device current.
struct DeviceSlot {
  void* ptr = nullptr;
  int num_cu = 0;
  int grid64 = 0, grid128 = 0;
};
std::mutex g_mu;
DeviceSlot g_slots[kMaxDevices];

size_t up256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

int fail(int code, const std::string& msg) {
  ent::set_free_error(msg);
  return code;
}

}  // namespace

extern "C" int ent_entropy_temperature_noalloc(const ent_config* cfg, int B, const float* logits,
                                               long long ld, ent_state st, float* h_out,
                                               float* temp_used, float* row_stats, void* stream) {
  // Host-side checks first: nothing below launches on a bad argument.
  int code;
  const std::string m = ent::config_error(cfg, &code);
  if (code != ENT_OK) return fail(code, "ent_entropy_temperature_noalloc: " + m);
  if (B < 0 || B > cfg->max_batch)
    return fail(ENT_E_INVAL, "ent_entropy_temperature_noalloc: B must be in [0, max_batch]");
  if (B == 0) {
    ent::set_free_error("");
    return ENT_OK;
  }
  if (!logits || !st.h_prev || !st.tau || !st.temp || !h_out || !temp_used)
    return fail(ENT_E_INVAL, "ent_entropy_temperature_noalloc: NULL required pointer");
  if (ld < cfg->vocab) return fail(ENT_E_INVAL, "ent_entropy_temperature_noalloc: ld < vocab");
  if (h_out == st.h_prev)
    return fail(ENT_E_INVAL, "ent_entropy_temperature_noalloc: h_out aliases h_prev");
  if (temp_used == st.temp)
    return fail(ENT_E_INVAL, "ent_entropy_temperature_noalloc: temp_used aliases temp");
  const int C = ent_row_stats_chunks(cfg->vocab);
  const bool est = ent::uses_estimate(*cfg);
  const size_t part_bytes = up256(static_cast<size_t>(B) * C * 3 * sizeof(float));
  const size_t tmax_bytes =
      est ? up256(static_cast<size_t>(B) * C * ent::kEstChunkThreads * sizeof(float)) : 0;
  const size_t flag_bytes = 256;
  if (part_bytes + tmax_bytes + flag_bytes > ENT_NOALLOC_SCRATCH_BYTES)
    return fail(ENT_E_UNSUPPORTED,
                "ent_entropy_temperature_noalloc: B * ceil(vocab / 4096) is too large for the "
                "static scratch (" + std::to_string(part_bytes + tmax_bytes + flag_bytes) +
                    " bytes needed, ENT_NOALLOC_SCRATCH_BYTES = " +
                    std::to_string(ENT_NOALLOC_SCRATCH_BYTES) + ")");

  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess)
    return fail(ENT_E_HIP, std::string("ent_entropy_temperature_noalloc: hipGetDevice: ") +
                               hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(ENT_E_UNSUPPORTED, "ent_entropy_temperature_noalloc: device index above 63");

  ent_ctx c;                 // host-side description of the launch; owns no device memory
  c.cfg = *cfg;
  c.device = dev;
  c.group = cfg->num_q_heads / cfg->num_kv_heads;
  c.chunks = C;
  {
    std::lock_guard<std::mutex> lk(g_mu);
    DeviceSlot& sl = g_slots[dev];
    if (!sl.ptr) {
      void* p = nullptr;
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess)
        return fail(ENT_E_HIP, std::string("ent_entropy_temperature_noalloc: hipGetSymbolAddress: ") +
                                   hipGetErrorString(e));
      int ncu = 0;
      e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
      if (e != hipSuccess)
        return fail(ENT_E_HIP, std::string("ent_entropy_temperature_noalloc: device query: ") +
                                   hipGetErrorString(e));
      ent_ctx probe;
      probe.cfg = *cfg;
      probe.num_cu = ncu;
      probe.cfg.head_dim = 64;
      sl.grid64 = ent::prologue_grid_size(&probe);
      probe.cfg.head_dim = 128;
      sl.grid128 = ent::prologue_grid_size(&probe);
      sl.num_cu = ncu;
      sl.ptr = p;
    }
    c.num_cu = sl.num_cu;
    c.prologue_grid = cfg->head_dim == 128 ? sl.grid128 : sl.grid64;
    unsigned char* base = static_cast<unsigned char*>(sl.ptr);
    c.dev_flags = reinterpret_cast<unsigned*>(base);
    c.ent_part = reinterpret_cast<float*>(base + flag_bytes);
    c.tmax = est ? reinterpret_cast<float*>(base + flag_bytes + part_bytes) : nullptr;
  }
  // Nothing in the array needs to start at zero: the chunk pass writes every
  // triple and maximum the merge reads, and no job of this pass raises the
  // flag word.
  e = ent::launch_entropy(&c, B, logits, ld, st, h_out, temp_used, row_stats, true,
                          static_cast<hipStream_t>(stream));
  if (e != hipSuccess)
    return fail(ENT_E_HIP, std::string("ent_entropy_temperature_noalloc launch: ") +
                               hipGetErrorString(e));
  ent::set_free_error("");
  return ENT_OK;
}
