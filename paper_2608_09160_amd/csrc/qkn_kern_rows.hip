// libqkn: the register-path kernels of the bf16 fused, apply and Phase A modes (the kernel templates are in qkn_kernels.h).

#include "qkn_kernels.h"

namespace qkn_dev {

const RowsFn kFusedTable[2][4][5] = {QKN_FULL_SET(FmtBf16, kFused, 0),
                                     QKN_FULL_SET(FmtBf16, kFused, 1)};
const RowsFn kApplyTable[2][4] = {QKN_ONE_SET(FmtBf16, kApply, 0), QKN_ONE_SET(FmtBf16, kApply, 1)};
const RowsFn kPartialTable[2][4] = {QKN_ONE_SET(FmtBf16, kPartial, 0),
                                    QKN_ONE_SET(FmtBf16, kPartial, 1)};

}  // namespace qkn_dev
