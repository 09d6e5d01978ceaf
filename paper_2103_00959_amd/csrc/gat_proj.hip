// The fused GAT aggregation with source scores projected from the gathered
// feature rows (k_gat with PROJ = true), instantiated apart from gat.hip so the
// two translation units compile in parallel.  The entry point is in gat.hip.
#include "gat_kernel.hpp"

namespace cogdl {
namespace {

template <typename TX, typename TY, bool BUF>
GatKernel pick_ch(int ch)
{
    constexpr int V = (int)(16 / sizeof(TX));
    if (ch == 1) return k_gat<TX, TY, V, 1, BUF, false, true>;
    if (ch == 2) return k_gat<TX, TY, V, 2, BUF, false, true>;
    return k_gat<TX, TY, V, 4, BUF, false, true>;
}

template <typename TX, bool BUF>
GatKernel pick_y(int ydt, int ch)
{
    if (ydt == COGDL_F32) return pick_ch<TX, float, BUF>(ch);
    if (ydt == COGDL_BF16) return pick_ch<TX, bf16_t, BUF>(ch);
    return pick_ch<TX, f16_t, BUF>(ch);
}

}  // namespace

GatKernel gat_pick_proj(int xdt, int ydt, int ch, bool buf)
{
    if (buf) {
        if (xdt == COGDL_F32) return pick_y<float, true>(ydt, ch);
        if (xdt == COGDL_BF16) return pick_y<bf16_t, true>(ydt, ch);
        return pick_y<f16_t, true>(ydt, ch);
    }
    if (xdt == COGDL_F32) return pick_y<float, false>(ydt, ch);
    if (xdt == COGDL_BF16) return pick_y<bf16_t, false>(ydt, ch);
    return pick_y<f16_t, false>(ydt, ch);
}

}  // namespace cogdl
