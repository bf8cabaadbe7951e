"""CPU oracle for the batched query-answering path (test infrastructure only)."""
