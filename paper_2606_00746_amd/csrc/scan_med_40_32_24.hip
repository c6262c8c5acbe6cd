// The register-streamed line scans at sides 40, 32 and 24 (a translation
// unit of their own so that the sides compile in parallel).
#include "scan_med.hpp"

namespace gspn {

template hipError_t med_fwd<40>(const Problem &, hipStream_t);
template hipError_t med_bwd<40>(const Problem &, hipStream_t);
template hipError_t med_fwd<32>(const Problem &, hipStream_t);
template hipError_t med_bwd<32>(const Problem &, hipStream_t);
template hipError_t med_fwd<24>(const Problem &, hipStream_t);
template hipError_t med_bwd<24>(const Problem &, hipStream_t);

}  // namespace gspn
