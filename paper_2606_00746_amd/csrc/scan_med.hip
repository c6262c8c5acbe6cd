// Dispatch of the register-streamed line scans (bf16 square planes of side
// 24 to 64, a multiple of 8) to the translation unit of each side; the
// kernels are in scan_med.hpp.
#include "launch.hpp"

namespace gspn {

bool med_supported(const Problem &p)
{
    // square planes whose side is a multiple of 8 between 24 and 64
    return p.dtype == 1 && p.H == p.W && p.H % 8 == 0 && p.H >= 24 && p.H <= 64;
}

hipError_t launch_fwd_med(const Problem &p, hipStream_t st)
{
    switch (p.H) {
    case 64: return med_fwd<64>(p, st);
    case 56: return med_fwd<56>(p, st);
    case 48: return med_fwd<48>(p, st);
    case 40: return med_fwd<40>(p, st);
    case 32: return med_fwd<32>(p, st);
    default: return med_fwd<24>(p, st);
    }
}

hipError_t launch_bwd_med(const Problem &p, hipStream_t st)
{
    switch (p.H) {
    case 64: return med_bwd<64>(p, st);
    case 56: return med_bwd<56>(p, st);
    case 48: return med_bwd<48>(p, st);
    case 40: return med_bwd<40>(p, st);
    case 32: return med_bwd<32>(p, st);
    default: return med_bwd<24>(p, st);
    }
}

}  // namespace gspn
