// The register-streamed line scans at side 64 (a translation unit of their own so that
// the sides compile in parallel).
#include "scan_med.hpp"

namespace gspn {

template hipError_t med_fwd<64>(const Problem &, hipStream_t);
template hipError_t med_bwd<64>(const Problem &, hipStream_t);

}  // namespace gspn
