// The fused GAT aggregation with source scores projected from the gathered
// feature rows (k_gat with PM = 1 or 2), instantiated apart from gat.hip so the
// two translation units compile in parallel.  The entry point is in gat.hip.
#include "gat_kernel.hpp"

namespace cogdl {
namespace {

template <typename TX, typename TY, bool BUF>
GatKernel pick_ch(int ch, bool dist)
{
    constexpr int V = (int)(16 / sizeof(TX));
    if (ch == 1) return dist ? k_gat<TX, TY, V, 1, BUF, false, 2> : k_gat<TX, TY, V, 1, BUF, false, 1>;
    if (ch == 2) return k_gat<TX, TY, V, 2, BUF, false, 1>;
    return k_gat<TX, TY, V, 4, BUF, false, 1>;
}

template <typename TX, bool BUF>
GatKernel pick_y(int ydt, int ch, bool dist)
{
    if (ydt == COGDL_F32) return pick_ch<TX, float, BUF>(ch, dist);
    if (ydt == COGDL_BF16) return pick_ch<TX, bf16_t, BUF>(ch, dist);
    return pick_ch<TX, f16_t, BUF>(ch, dist);
}

}  // namespace

GatKernel gat_pick_proj(int xdt, int ydt, int ch, bool buf, bool dist)
{
    if (buf) {
        if (xdt == COGDL_F32) return pick_y<float, true>(ydt, ch, dist);
        if (xdt == COGDL_BF16) return pick_y<bf16_t, true>(ydt, ch, dist);
        return pick_y<f16_t, true>(ydt, ch, dist);
    }
    if (xdt == COGDL_F32) return pick_y<float, false>(ydt, ch, dist);
    if (xdt == COGDL_BF16) return pick_y<bf16_t, false>(ydt, ch, dist);
    return pick_y<f16_t, false>(ydt, ch, dist);
}

}  // namespace cogdl
