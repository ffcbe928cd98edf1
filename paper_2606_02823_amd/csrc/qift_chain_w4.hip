// Persistent decode-chain kernel for the W4 weight format (qift_chain.h; one instance per format so
// that the instances compile in parallel).
#include "qift_chain.h"

namespace qift {

hipError_t launch_chain_w4(const ChainDesc* links, int n_links, const uint16_t* x0, int M, int Kmax, int region0,
                          int grid, unsigned* counters, hipStream_t s) {
  return launch_chain_fmt<mma::FMT_W4>(links, n_links, x0, M, Kmax, region0, grid, counters, s);
}

}  // namespace qift
