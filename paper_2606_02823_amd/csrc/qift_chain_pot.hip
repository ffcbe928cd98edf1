// Persistent decode-chain kernel for the POT weight format (qift_chain.h; one instance per format so
// that the instances compile in parallel).
#include "qift_chain.h"

namespace qift {

hipError_t launch_chain_pot(const ChainDesc* links, int n_links, const uint16_t* x0, int M, int Kmax, bool any_long,
                          int grid, unsigned* counters, hipStream_t s) {
  return launch_chain_fmt<mma::FMT_POT>(links, n_links, x0, M, Kmax, any_long, grid, counters, s);
}

}  // namespace qift
