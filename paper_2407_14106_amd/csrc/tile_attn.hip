// Dense-tile attention on the matrix cores (placeholder until the MFMA kernels land).
#include "tile_attn.h"

namespace gt {

template <typename T, int D, int H>
gt_status tile_fwd(const gt_tiles*, const T*, const T*, const T*, float, TilePartials, hipStream_t) {
    return fail(GT_ERR_UNSUPPORTED, "dense tiles are not supported yet");
}

template <typename T, int D, int H>
gt_status tile_bwd_dq(const gt_tiles*, const T*, const T*, const T*, const T*, const T*, const float*, float*, float,
                      TilePartials, hipStream_t) {
    return fail(GT_ERR_UNSUPPORTED, "dense tiles are not supported yet");
}

template <typename T, int D, int H>
gt_status tile_bwd_dkdv(const gt_tiles*, const T*, const T*, const T*, const T*, const float*, const float*, float,
                        TilePartials, TilePartials, hipStream_t) {
    return fail(GT_ERR_UNSUPPORTED, "dense tiles are not supported yet");
}

#define GT_INST(T, D, H)                                                                                          \
    template gt_status tile_fwd<T, D, H>(const gt_tiles*, const T*, const T*, const T*, float, TilePartials,      \
                                         hipStream_t);                                                            \
    template gt_status tile_bwd_dq<T, D, H>(const gt_tiles*, const T*, const T*, const T*, const T*, const T*,    \
                                            const float*, float*, float, TilePartials, hipStream_t);              \
    template gt_status tile_bwd_dkdv<T, D, H>(const gt_tiles*, const T*, const T*, const T*, const T*,            \
                                              const float*, const float*, float, TilePartials, TilePartials,      \
                                              hipStream_t);
#define GT_INST_H(T, D) GT_INST(T, D, 1) GT_INST(T, D, 2) GT_INST(T, D, 4) GT_INST(T, D, 8) GT_INST(T, D, 16)
GT_INST_H(uint16_t, 32)
GT_INST_H(uint16_t, 64)
GT_INST_H(float, 32)
GT_INST_H(float, 64)

}  // namespace gt
