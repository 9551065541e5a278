// libqkn: the bf16 waiting and publishing kernels (the kernel templates are in qkn_kernels.h).

#include "qkn_kernels.h"

namespace qkn_dev {

// The publish-ahead schedules (2..4) hold extra tokens in registers; with Q
// and K rows both of 8 chunks per lane they spill to scratch, so those slots
// are left empty and the host takes the pipelined schedule there instead.
#define QKN_AHEAD_SET(S)                                                        \
  {QKN_ROW_SET(FmtBf16, kFusedWait, 1, S), QKN_ROW_SET(FmtBf16, kFusedWait, 2, S), \
   QKN_ROW_SET(FmtBf16, kFusedWait, 4, S),                                       \
   {qkn_rows<FmtBf16, 8, 0, kFusedWait, S>, qkn_rows<FmtBf16, 8, 1, kFusedWait, S>, \
    qkn_rows<FmtBf16, 8, 2, kFusedWait, S>, qkn_rows<FmtBf16, 8, 4, kFusedWait, S>, nullptr}}

const RowsFn kFusedWaitTable[5][4][5] = {
    QKN_FULL_SET(FmtBf16, kFusedWait, 0), QKN_FULL_SET(FmtBf16, kFusedWait, 1),
    QKN_AHEAD_SET(2), QKN_AHEAD_SET(3), QKN_AHEAD_SET(4)};
const RowsFn kPublishTable[4] = QKN_ONE_SET(FmtBf16, kPublish, 0);

}  // namespace qkn_dev
