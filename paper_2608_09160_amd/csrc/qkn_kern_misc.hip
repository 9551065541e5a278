// libqkn: the FP8 register-path kernels, the wide-row kernels and the general kernels (the kernel templates are in qkn_kernels.h).

#include "qkn_kernels.h"

namespace qkn_dev {

const RowsFn kFusedTable8[4][5] = QKN_FULL_SET8(kFused, 0);
const RowsFn kApplyTable8[4] = QKN_ONE_SET8(kApply, 0);
const RowsFn kPartialTable8[4] = QKN_ONE_SET8(kPartial, 0);
const GenericFn kGenericTable[2][3] = {
    {qkn_generic<FmtBf16, kFused>, qkn_generic<FmtBf16, kApply>, qkn_generic<FmtBf16, kPartial>},
    {qkn_generic<FmtFp8, kFused>, qkn_generic<FmtFp8, kApply>, qkn_generic<FmtFp8, kPartial>}};
const RowsFn kWideTable[2][2][3][5] = {
    {{QKN_WIDE_SET(FmtBf16, 16, kFused), QKN_WIDE_SET(FmtBf16, 16, kApply),
      QKN_WIDE_SET(FmtBf16, 16, kPartial)},
     {QKN_WIDE_SET(FmtBf16, 32, kFused), QKN_WIDE_SET(FmtBf16, 32, kApply),
      QKN_WIDE_SET(FmtBf16, 32, kPartial)}},
    {{QKN_WIDE_SET8(8, kFused), QKN_WIDE_SET8(8, kApply), QKN_WIDE_SET8(8, kPartial)},
     {QKN_WIDE_SET8(16, kFused), QKN_WIDE_SET8(16, kApply), QKN_WIDE_SET8(16, kPartial)}}};

}  // namespace qkn_dev
