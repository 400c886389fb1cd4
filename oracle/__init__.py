"""CPU oracle for GDN draft-tree verification (test infrastructure only)."""
