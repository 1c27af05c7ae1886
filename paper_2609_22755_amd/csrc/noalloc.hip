// Device scratch of the allocation-free backward entry point
// (nsp_varlen_attn_bwd_noalloc): one file-scope device array, which every GPU
// the library runs on holds from the module's load to the end of the process.
// Host code never uses the array's name as an address: the device address of
// each GPU's copy is looked up once per device, with that device current, and
// kept.
#include <mutex>
#include <unordered_map>

#include "nsp_internal.hpp"

namespace nsp {
namespace {

__device__ __align__(256) char scratch[kScratchBytes];

std::mutex g_scratch_mu;
std::unordered_map<int, char *> g_scratch_ptr;   // device -> address of its copy

}  // namespace

hipError_t noalloc_scratch(char **ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  auto it = g_scratch_ptr.find(dev);
  if (it == g_scratch_ptr.end()) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    it = g_scratch_ptr.emplace(dev, static_cast<char *>(p)).first;
  }
  *ptr = it->second;
  return hipSuccess;
}

}  // namespace nsp
