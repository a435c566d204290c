"""libmoe for MI355X: the MoE layer forward on one GPU's TP or EP share.

The compute lives in libmoe.so (HIP kernels for gfx950 behind the C ABI in
include/libmoe.h); this package only binds it.
"""
from .binding import (MoeError, MoeLayer, combine, ffn_workspace_size, grouped_ffn,  # noqa: F401
                     grouped_ffn_shared, lib, ExpertSlots, reshard_experts, EP_TO_TP, TP_TO_EP,
                     kv_slots, kv_move, SwitchPolicy, partition_requests, kv_fits, policy_crossover,
                     MODE_TP, MODE_EP, STAY, SWITCH, SWITCH_CANCELLED,
                     permute, permute_workspace_size, layer_workspace_size, route, timing_enable, timing_read,
                     timing_reset, timing_device_enable, timing_device_clear,
                     timing_device_reset, timing_device_read, calib_mfma)

__all__ = ["MoeError", "MoeLayer", "route", "permute", "grouped_ffn", "grouped_ffn_shared", "combine", "lib",
           "permute_workspace_size", "ffn_workspace_size", "layer_workspace_size", "ExpertSlots", "reshard_experts", "EP_TO_TP",
           "TP_TO_EP", "kv_slots", "kv_move", "SwitchPolicy", "partition_requests", "kv_fits",
           "policy_crossover", "MODE_TP", "MODE_EP", "STAY", "SWITCH", "SWITCH_CANCELLED", "timing_enable",
           "timing_read", "timing_reset", "timing_device_enable", "timing_device_clear", "timing_device_reset",
           "timing_device_read", "calib_mfma"]
