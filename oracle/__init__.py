"""CPU oracle for the Mixture-of-Translators KV-cache translation.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg use it.  The GPU library never imports it, and it never
imports the GPU library.  It follows the paper's Definition
"Mixture-of-Translators" (Sec. 3, Eq. mot_definition) literally, in double
precision; see ``mot_oracle.c`` for the step-by-step statement.
"""
from .oracle import (OracleDims, build_oracle, oracle_translate, oracle_rows,
                     oracle_depth_ratio_map, oracle_lib_path, oracle_restore_kv,
                     oracle_topS_select, oracle_replay_attention, oracle_topS_rows,
                     oracle_replay_attention_rows, oracle_backbone_translate, oracle_backbone_param_count,
                     oracle_usage, oracle_usage_stats, oracle_backbone_window,
                     oracle_backbone_window_param_count)

__all__ = ["OracleDims", "build_oracle", "oracle_translate", "oracle_rows",
           "oracle_depth_ratio_map", "oracle_lib_path", "oracle_restore_kv",
           "oracle_topS_select", "oracle_replay_attention", "oracle_topS_rows",
           "oracle_replay_attention_rows", "oracle_backbone_translate", "oracle_backbone_param_count",
           "oracle_usage", "oracle_usage_stats", "oracle_backbone_window",
           "oracle_backbone_window_param_count"]
