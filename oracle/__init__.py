"""CPU oracle for the TeraPipe stage and slicer -- TEST INFRASTRUCTURE ONLY.

Only tests/, the smoke check and the CPU-baseline leg of the benchmark may use
this package.  It never imports the GPU library and the GPU library never
imports it.
"""
from .oracle import (OracleStage, batch_split, cost_table_from_model, exhaustive_batch_split,
                     integer_partitions, joint_slicing, dp_optimal_slicing, eq5_latency,
                     exhaustive_optimal, fit_ctx_model, gelu, gelu_grad, load_library,
                     slice_flops, sequence_flops, paper_tflops_per_gpu, PARAM_NAMES)

__all__ = ["OracleStage", "batch_split", "exhaustive_batch_split", "integer_partitions",
           "joint_slicing", "cost_table_from_model", "fit_ctx_model", "dp_optimal_slicing", "eq5_latency", "exhaustive_optimal", "gelu",
           "gelu_grad", "load_library", "slice_flops", "sequence_flops", "paper_tflops_per_gpu",
           "PARAM_NAMES"]
