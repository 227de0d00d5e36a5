// Library-internal declarations shared by the HIP sources of libdpc.
#ifndef DPC_INTERNAL_H
#define DPC_INTERNAL_H

// DPC_OK if nothing was raised since the last call, else DPC_EHIP (the HIP
// error is kept for dpc_last_hip_error() of this thread).
int dpc_internal_launch_status();

#endif  // DPC_INTERNAL_H
