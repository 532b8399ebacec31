// Instances of the fused pass: 4-row items in blocks of kBigBlock threads.

#include "sdb_fused.h"

namespace sdb {

const void* pick_fused_big(int ipt, int terminal) {
    if (ipt == 1) { SDB_FUSED_TERMINALS(4, 1, false, kBigBlock, 0) }
    if (ipt == 2) { SDB_FUSED_TERMINALS(4, 2, false, kBigBlock, 0) }
    return nullptr;
}

}  // namespace sdb
