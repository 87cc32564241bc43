"""CPU oracle for the ExFold folded MoE layer (test infrastructure only)."""
