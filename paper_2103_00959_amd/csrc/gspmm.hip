// Instantiations of the generalized SpMM gather kernel (section 2.2, Eq. 1)
// for the reduce / compute pairs beyond the sum of products: max of
// products, and sum or max of x + bsign * val (add, subtract).  Kept in a
// translation unit of their own so that the library builds in parallel.
#include "spmm_kernel.hpp"

namespace cogdl {

SpmmKernel gspmm_pick(bool maxr, bool addop, int xdt, int ydt, int vec, int ch, bool buf)
{
    if (maxr && addop) return spmm_pick<true, true>(xdt, ydt, vec, ch, buf);
    if (maxr) return spmm_pick<true, false>(xdt, ydt, vec, ch, buf);
    if (addop) return spmm_pick<false, true>(xdt, ydt, vec, ch, buf);
    return nullptr;
}

}  // namespace cogdl
