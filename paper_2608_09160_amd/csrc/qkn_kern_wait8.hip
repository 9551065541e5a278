// libqkn: the FP8 waiting and publishing kernels (the kernel templates are in qkn_kernels.h).

#include "qkn_kernels.h"

namespace qkn_dev {

const RowsFn kFusedWaitTable8[5][4][5] = {
    QKN_FULL_SET8(kFusedWait, 0), QKN_FULL_SET8(kFusedWait, 1), QKN_FULL_SET8(kFusedWait, 2),
    QKN_FULL_SET8(kFusedWait, 3), QKN_FULL_SET8(kFusedWait, 4)};
const RowsFn kPublishTable8[4] = QKN_ONE_SET8(kPublish, 0);

}  // namespace qkn_dev
