// Persistent decode-chain kernel for the MNZ weight format (qift_chain.h; one instance per format so
// that the instances compile in parallel).
#include "qift_chain.h"

namespace qift {

hipError_t launch_chain_mnz(const ChainDesc* links, int n_links, const uint16_t* x0, int M, int Kmax, int region0,
                          int grid, unsigned* counters, hipStream_t s) {
  return launch_chain_fmt<mma::FMT_MNZ>(links, n_links, x0, M, Kmax, region0, grid, counters, s);
}

}  // namespace qift

#ifdef QIFT_CHAIN_STAMPS
// The diagnostic build's reader of the MNZ chain's phase stamps (qift_chain.h): bytes of
// g_chain_stamps into host memory.  Not part of the product library's interface.
extern "C" int qift_chain_stamps_read(void* host, size_t bytes) {
  if (bytes > sizeof(qift::g_chain_stamps)) return -1;
  return (int)hipMemcpyFromSymbol(host, HIP_SYMBOL(qift::g_chain_stamps), bytes, 0, hipMemcpyDeviceToHost);
}
#endif
