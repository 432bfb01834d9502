"""MI355X-native batched VQC statevector engine (VQCSim hot path)."""
